"""Benchmark: routed token-expert pairs per second of the EW forward on one GPU.

One step is one tg_ew_forward call (gating, ERT remap and dispatch, grouped
SwiGLU expert FFN, combine) over the Mixtral-shaped workload: T=4096 tokens,
d=4096, E=8 experts, top-2, I=14336, 8 primary + 2 shadow slots, synthetic
bf16 inputs already resident in HBM. Prints one JSON line; its "workloads"
key carries the same measurement, compact, for the DeepSeek-V3 expert share
(T=16384, d=7168, 256 experts, top-8, I=2048, 32 + 8 slots), its skewed
failover variant and the decode-size batch (T=128).

  python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload mixtral]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
RIDGE_FLOP_PER_BYTE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
STAGES = ["gate", "dispatch", "ffn_gateup", "ffn_down", "combine"]
GEMM_SRC = [os.path.join(ROOT, "paper_2601_01310_amd", "csrc", f)
            for f in ("grouped_gemm.hip", "tg_device.h")]
TRAFFIC = os.path.join(ROOT, "profiles", "gemm_traffic.json")


def kernel_source_hash(paths) -> str:
    """sha256 of the kernel sources with comments and blank lines removed:
    it changes when the code changes, not when a comment does."""
    import hashlib
    import re
    out = []
    for f in paths:
        text = open(f, encoding="utf-8").read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for line in text.splitlines():
            line = re.sub(r"//.*", "", line).rstrip()
            if line.strip():
                out.append(line)
    return hashlib.sha256("\n".join(out).encode()).hexdigest()


def measured_traffic(workload: str):
    """HBM-side bytes per dispatch of the gate/up GEMM on this workload from
    the committed rocprofv3 FETCH_SIZE / WRITE_SIZE runs, or None when they
    were not taken on it or were taken before the kernel source last
    changed."""
    try:
        rec = json.load(open(TRAFFIC))
    except (OSError, ValueError):
        return None
    sha = kernel_source_hash(GEMM_SRC)
    w = rec.get("workloads", {}).get(workload)
    if rec.get("source_sha256") != sha or not w:
        return None
    return w["gateup"]["traffic_bytes_per_dispatch"]


class HipEvents:
    """hipEvent_t handles through the HIP runtime's C API (timing only)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            ev = ctypes.c_void_p()
            if self.hip.hipEventCreate(ctypes.byref(ev)) != 0:
                raise RuntimeError("hipEventCreate failed")
            out.append(ev.value)
        return out

    def record(self, ev, stream):
        if self.hip.hipEventRecord(ctypes.c_void_p(ev), ctypes.c_void_p(stream.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, evs):
        for e in evs:
            self.hip.hipEventDestroy(ctypes.c_void_p(e))


def cpu_baseline(wl, n_tokens: int = 1536):
    """The CPU oracle, as it stands, on a bounded sample of the workload:
    the full forward of ``n_tokens`` seeded tokens (their routed pairs)."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    from oracle import moe_ew as O

    def host(t):
        t = t.detach().cpu().contiguous()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()

    x, ert, alive = host(wl.x), host(wl.ert), host(wl.alive)
    wg = None if wl.wg is None else host(wl.wg)
    logits = None if wl.logits is None else host(wl.logits)
    w13 = [host(wl.w13[s]) for s in range(wl.S)]
    w2 = [host(wl.w2[s]) for s in range(wl.S)]
    n_tokens = min(n_tokens, wl.T)  # a decode batch is smaller than the sample: take all of it
    toks = sorted(np.random.default_rng(0).choice(wl.T, size=n_tokens, replace=False).tolist())
    t0 = time.perf_counter()
    _, _, ps, _ = O.ew_forward_tokens(toks, x, wg, logits, wl.k, ert, alive,
                                      lambda s: w13[s], lambda s: w2[s])
    dt = time.perf_counter() - t0
    pairs = int((ps >= 0).sum())
    blas = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    cores, model = host_cpu()
    return {"value": pairs / dt, "unit": "routed pairs/s", "cores": int(min(blas, cores)),
            "kind": "oracle",
            "sample": f"{n_tokens} seeded tokens of the workload ({pairs} routed pairs), float64 "
                      f"per-token oracle incl. widening the touched slots' bf16 weights; {dt:.1f} s",
            "host_cores": cores, "blas_threads": int(blas), "cpu_model": model}


def host_cpu():
    """CPUs this process may run on (nproc) and the CPU model name."""
    try:
        cores = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        cores = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return cores, model


def _ffn_buffers(d, I, S, max_rows, dev, seed=0):
    import torch
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    x = (torch.randn((max_rows, d), generator=g, device=dev)).to(torch.bfloat16)
    w13 = (torch.randn((S, 2 * I, d), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    w2 = (torch.randn((S, d, I), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    h = torch.empty((max_rows, I), dtype=torch.bfloat16, device=dev)
    y = torch.empty((max_rows, d), dtype=torch.bfloat16, device=dev)
    return x, w13, w2, h, y


def _offsets(counts, dev):
    import torch
    off = [0]
    for c in counts:
        off.append(off[-1] + c)
    return torch.tensor(off, dtype=torch.int32, device=dev)


def expert_batch_knee(dev, reps=20):
    """Expert FFN latency and throughput against the expert batch size (the
    paper's expert-batch-size knee, App. B), through tg_expert_ffn_grouped with
    all rows in one slot. Slots rotate over 8 copies so the weights come from
    HBM, not from the 256 MB Infinity Cache. Each size is timed with the
    launch's own tile choice and with each tile height forced."""
    import torch

    from paper_2601_01310_amd import tg

    hip = HipEvents()
    out = []
    for name, d, I in (("mixtral expert", 4096, 14336), ("deepseek-v3 expert", 7168, 2048)):
        S = 8
        Ms = [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096]
        x, w13, w2, h, y = _ffn_buffers(d, I, S, max(Ms), dev)
        for M in Ms:
            offs = [_offsets([M if s == j else 0 for s in range(S)], dev) for j in range(S)]

            def timed(policy):
                from ctypes import c_void_p
                with tg.tile_policy(policy):
                    for j in range(3):
                        tg.tg_expert_ffn_grouped(x, offs[j % S], S, M, w13, w2, d, I, h, y)
                    ev = hip.create(2)
                    torch.cuda.synchronize()
                    stream = c_void_p(torch.cuda.current_stream().cuda_stream)
                    hip.hip.hipEventRecord(c_void_p(ev[0]), stream)
                    for j in range(reps):
                        tg.tg_expert_ffn_grouped(x, offs[j % S], S, M, w13, w2, d, I, h, y)
                    hip.hip.hipEventRecord(c_void_p(ev[1]), stream)
                    torch.cuda.synchronize()
                us = hip.elapsed_ms(ev[0], ev[1]) * 1e3 / reps
                hip.destroy(ev)
                return us

            us = timed(tg.TILES_AUTO)
            us_small, us_full = timed(tg.TILES_SMALL), timed(tg.TILES_FULL)
            flops = 6.0 * d * I * M
            wbytes = 3.0 * d * I * 2
            rec = dict(expert=name, rows=M, us=us, tflops=flops / us / 1e6,
                       weight_tbps=wbytes / us / 1e6, us_per_row=us / M,
                       us_32row_tiles=us_small, us_256row_tiles=us_full)
            out.append(rec)
            print(json.dumps(rec), flush=True)
        del x, w13, w2, h, y
        torch.cuda.empty_cache()
    return out


def shadow_interference(dev, reps=20):
    """Loaded-but-idle shadow slot vs a single expert vs two experts run
    concurrently on two streams with the same total batch (App. D)."""
    import torch
    from ctypes import c_void_p

    from paper_2601_01310_amd import tg

    hip = HipEvents()
    d, I, M = 4096, 14336, 512
    S = 8
    x, w13, w2, h, y = _ffn_buffers(d, I, S, M, dev)
    h2 = torch.empty_like(h)
    y2 = torch.empty_like(y)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()

    def timed(fn):
        for j in range(3):
            fn(j)
        torch.cuda.synchronize()
        ev = hip.create(2)
        cur = torch.cuda.current_stream()
        hip.hip.hipEventRecord(c_void_p(ev[0]), c_void_p(cur.cuda_stream))
        s1.wait_stream(cur)
        s2.wait_stream(cur)
        for j in range(reps):
            fn(j)
        cur.wait_stream(s1)
        cur.wait_stream(s2)
        hip.hip.hipEventRecord(c_void_p(ev[1]), c_void_p(cur.cuda_stream))
        torch.cuda.synchronize()
        us = hip.elapsed_ms(ev[0], ev[1]) * 1e3 / reps
        hip.destroy(ev)
        return us

    one = [_offsets([M if s == j % 4 else 0 for s in range(4)], dev) for j in range(4)]
    # slot j%4 active with M rows, plus 4 loaded shadow slots (copies) that stay idle
    with_shadow = [_offsets([M if s == j % 4 else 0 for s in range(S)], dev) for j in range(4)]
    half_a = [_offsets([M // 2 if s == (2 * j) % 8 else 0 for s in range(S)], dev) for j in range(4)]
    half_b = [_offsets([M // 2 if s == (2 * j + 1) % 8 else 0 for s in range(S)], dev) for j in range(4)]
    grouped = [_offsets([M // 2 if s in ((2 * j) % 8, (2 * j + 1) % 8) else 0 for s in range(S)], dev)
               for j in range(4)]

    def single(j):
        tg.tg_expert_ffn_grouped(x, one[j % 4], 4, M, w13, w2, d, I, h, y)

    def shadow_loaded(j):
        tg.tg_expert_ffn_grouped(x, with_shadow[j % 4], S, M, w13, w2, d, I, h, y)

    def concurrent(j):
        with torch.cuda.stream(s1):
            tg.tg_expert_ffn_grouped(x, half_a[j % 4], S, M // 2, w13, w2, d, I, h, y, stream=s1)
        with torch.cuda.stream(s2):
            tg.tg_expert_ffn_grouped(x, half_b[j % 4], S, M // 2, w13, w2, d, I, h2, y2, stream=s2)

    def two_in_one_launch(j):
        tg.tg_expert_ffn_grouped(x, grouped[j % 4], S, M, w13, w2, d, I, h, y)

    cases = (("single_expert_us", single), ("single_plus_idle_shadows_us", shadow_loaded),
             ("two_experts_two_streams_us", concurrent),
             ("two_experts_one_grouped_launch_us", two_in_one_launch))
    # Two passes over all cases; the first brings clocks and caches to a
    # steady state and is discarded.
    for _ in range(2):
        res = {"rows_total": M, "expert": "mixtral expert (d=4096, I=14336)"}
        for name, fn in cases:
            res[name] = timed(fn)
    print(json.dumps(res), flush=True)
    return res


def replay_cost(wl, steps, warmup):
    """Cost of replaying the pairs of the workload's failed primaries on
    their shadows after a completed forward (§5.1), against the forward
    itself; HIP events around each call."""
    import torch
    from ctypes import c_void_p

    from paper_2601_01310_amd import tg

    hip = HipEvents()
    stream = torch.cuda.current_stream()
    f = tg.EwForward(wl, keep_y=True)
    alive1 = wl.alive_after_failure()

    def timed(fn):
        for _ in range(warmup):
            fn()
        ev = hip.create(2 * steps)
        torch.cuda.synchronize()
        for i in range(steps):
            hip.hip.hipEventRecord(c_void_p(ev[2 * i]), c_void_p(stream.cuda_stream))
            fn()
            hip.hip.hipEventRecord(c_void_p(ev[2 * i + 1]), c_void_p(stream.cuda_stream))
        torch.cuda.synchronize()
        us = sorted(hip.elapsed_ms(ev[2 * i], ev[2 * i + 1]) * 1e3 for i in range(steps))
        hip.destroy(ev)
        return us[len(us) // 2]

    fwd_us = timed(lambda: f(stream))
    f(stream)
    rep_us = timed(lambda: f.replay(alive1, stream))
    _, n_rep, _ = f.replay(alive1, stream)
    torch.cuda.synchronize()
    res = {"workload": wl.name, "failed_slots": int((wl.alive != alive1).sum()),
           "pairs_replayed": int(n_rep[0]), "routed_pairs": int(f.slot_offsets[-1]),
           "forward_us_p50": fwd_us, "replay_us_p50": rep_us}
    print(json.dumps(res), flush=True)
    return res


def partial_batch_cost(wl, steps, warmup, n_aws=8, late=(3,)):
    """EW-side partial batch (§5.2): the workload's tokens arrive from n_aws
    attention workers in equal chunks; the AWs in ``late`` never deliver and
    the trigger fires on the minimum batch (the other AWs' rows). Times the
    trigger alone, trigger + forward on the partial batch, and the forward
    on the full batch (HIP events, p50)."""
    import torch
    from ctypes import c_void_p

    from paper_2601_01310_amd import tg

    dev = wl.x.device
    hip = HipEvents()
    stream = torch.cuda.current_stream()
    bounds = [wl.T * a // n_aws for a in range(n_aws + 1)]
    chunk_rows = torch.tensor(bounds, dtype=torch.int32, device=dev)
    delivered = torch.tensor([0 if a in late else 1 for a in range(n_aws)], dtype=torch.int32,
                             device=dev)
    alive = torch.ones(n_aws, dtype=torch.uint8, device=dev)
    min_rows = sum(bounds[a + 1] - bounds[a] for a in range(n_aws) if a not in late)
    tv = torch.empty(wl.T, dtype=torch.uint8, device=dev)
    st = torch.empty(4, dtype=torch.int32, device=dev)
    part = tg.EwForward(wl, token_valid=tv)
    full = tg.EwForward(wl)

    def trigger():
        tg.tg_batch_trigger(delivered, alive, chunk_rows, n_aws, wl.T, min_rows, 1000, tv, st,
                            stream)

    def both():
        trigger()
        part(stream)

    def timed(fn):
        for _ in range(warmup):
            fn()
        ev = hip.create(2 * steps)
        torch.cuda.synchronize()
        for i in range(steps):
            hip.hip.hipEventRecord(c_void_p(ev[2 * i]), c_void_p(stream.cuda_stream))
            fn()
            hip.hip.hipEventRecord(c_void_p(ev[2 * i + 1]), c_void_p(stream.cuda_stream))
        torch.cuda.synchronize()
        us = sorted(hip.elapsed_ms(ev[2 * i], ev[2 * i + 1]) * 1e3 for i in range(steps))
        hip.destroy(ev)
        return us[len(us) // 2]

    res = {"workload": wl.name, "aws": n_aws, "late_aws": list(late),
           "trigger_us_p50": timed(trigger), "trigger_plus_partial_forward_us_p50": timed(both),
           "full_forward_us_p50": timed(lambda: full(stream))}
    s = st.cpu().tolist()
    res.update({"condition": s[0], "rows_in_batch": s[1], "aws_in_batch": s[2],
                "pairs_partial": int(part.slot_offsets[-1]), "pairs_full": int(full.slot_offsets[-1])})
    print(json.dumps(res), flush=True)
    return res


def checkpoint_cost(wl, steps, warmup):
    """KV-segment checkpoint of one decode step (§6.1; Mixtral segments of
    2 * 8 KV heads * 128 * 2 bytes, App. C) for 128 requests over 32 layers
    into pinned host memory: its time alone, and the EW forward's time alone
    and with the checkpoint running on a second stream."""
    import numpy as np
    import torch
    from ctypes import c_void_p

    from paper_2601_01310_amd import tg

    dev = wl.x.device
    hip = HipEvents()
    main_s = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    seg, layers, requests, max_len = 4096, 32, 128, 64
    size = layers * requests * max_len * seg
    kv = torch.empty(size, dtype=torch.uint8, device=dev)
    kv.random_(0, 256)
    store = torch.empty(size, dtype=torch.uint8, pin_memory=True)
    log_cap = layers * requests
    log = torch.zeros(log_cap * 3, dtype=torch.int64, pin_memory=True)
    commit = torch.zeros(1, dtype=torch.int64, pin_memory=True)
    pos = 7
    offs = np.array([((l * requests + r) * max_len + pos) * seg for r in range(requests)
                     for l in range(layers)], dtype=np.int64)
    n = len(offs)
    od = torch.from_numpy(offs).to(dev)
    bd = torch.full((n,), seg, dtype=torch.int32, device=dev)
    f = tg.EwForward(wl)
    seq = [0]

    blocks = [0]

    def ckpt(stream):
        tg.tg_kv_checkpoint(kv, size, od, bd, n, seq[0], store, log, log_cap, commit, stream,
                            max_blocks=blocks[0])
        seq[0] += n

    def timed(fn, stream):
        for _ in range(warmup):
            fn()
        ev = hip.create(2 * steps)
        torch.cuda.synchronize()
        for i in range(steps):
            hip.hip.hipEventRecord(c_void_p(ev[2 * i]), c_void_p(stream.cuda_stream))
            fn()
            hip.hip.hipEventRecord(c_void_p(ev[2 * i + 1]), c_void_p(stream.cuda_stream))
        torch.cuda.synchronize()
        us = sorted(hip.elapsed_ms(ev[2 * i], ev[2 * i + 1]) * 1e3 for i in range(steps))
        hip.destroy(ev)
        return us[len(us) // 2]

    def both():
        side.wait_stream(main_s)
        ckpt(side)
        f(main_s)
        main_s.wait_stream(side)

    fwd_us = timed(lambda: f(main_s), main_s)
    paths = {}
    for g in (8, 16, 32):
        blocks[0] = g
        ck_us = timed(lambda: ckpt(main_s), main_s)
        both_us = timed(both, main_s)
        paths[f"kernel_{g}_blocks"] = {
            "checkpoint_us_p50": ck_us, "checkpoint_gbps": n * seg / ck_us / 1e3,
            "forward_with_concurrent_checkpoint_us_p50": both_us}
    # The same batch is strided (pitch = max_len segments): copy engine.
    first, pitch = pos * seg, max_len * seg

    def strided(stream):
        tg.tg_kv_checkpoint_strided(kv, size, first, pitch, seg, n, seq[0], store, log, log_cap,
                                    commit, stream)
        seq[0] += n

    def both_strided():
        side.wait_stream(main_s)
        strided(side)
        f(main_s)
        main_s.wait_stream(side)

    ck_us = timed(lambda: strided(main_s), main_s)
    paths["copy_engine_strided"] = {
        "checkpoint_us_p50": ck_us, "checkpoint_gbps": n * seg / ck_us / 1e3,
        "forward_with_concurrent_checkpoint_us_p50": timed(both_strided, main_s)}
    torch.cuda.synchronize()
    res = {"workload": wl.name, "segments": n, "segment_bytes": seg,
           "checkpoint_bytes": n * seg, "forward_us_p50": fwd_us, "paths": paths,
           "commit": int(commit[0])}
    print(json.dumps(res), flush=True)
    return res


def measured_peaks(dev):
    """What this GPU sustains on plain library work, as references next to
    the datasheet peaks: a large bf16 GEMM (hipBLASLt through torch), a bf16
    matrix-vector product over a 4 GiB matrix (weight streaming from HBM,
    the decode workload's access pattern) and a 2 GiB device copy (read +
    write). The HBM reference is the better of the last two."""
    import torch

    def best_ms(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            best = min(best, a.elapsed_time(b))
        return best

    # The Mixtral gate/up projection of 8192 routed rows as ONE dense GEMM
    # (8192 x 4096 x 28672): what the vendor library reaches on this work
    # without any grouping.
    M, K, N = 8192, 4096, 28672
    x = torch.randn(M, K, device=dev).to(torch.bfloat16)
    y = torch.randn(K, N, device=dev).to(torch.bfloat16)
    gemm = 2.0 * M * K * N / (best_ms(lambda: torch.matmul(x, y)) * 1e-3) / 1e12
    del x, y
    wmat = torch.randn(65536, 32768, device=dev).to(torch.bfloat16)  # 4 GiB
    vec = torch.randn(32768, device=dev).to(torch.bfloat16)
    read = wmat.numel() * 2 / (best_ms(lambda: torch.mv(wmat, vec)) * 1e-3) / 1e12
    del wmat, vec
    src = torch.ones(1 << 29, dtype=torch.float32, device=dev)  # 2 GiB
    dst = torch.empty_like(src)
    copy = 2 * src.numel() * 4 / (best_ms(lambda: dst.copy_(src)) * 1e-3) / 1e12
    del src, dst
    torch.cuda.empty_cache()
    return {"bf16_gemm_tflops": gemm, "hbm_read_tbps": read, "hbm_copy_tbps": copy,
            "how": "torch.matmul 8192x4096 @ 4096x28672 bf16; torch.mv over a 65536x32768 "
                   "bf16 matrix (4 GiB read); copy of 2 GiB (read + write bytes); best of 5"}


OTHER_WORKLOADS = ["dsv3_share", "dsv3_skew", "dsv3_decode"]
FAILOVER_BLOCKS = 8          # healthy / rerouted blocks, interleaved
FAILOVER_BLOCK_STEPS = 20    # at least this many steps per block


def _pct(v, q):
    v = sorted(v)
    return v[min(len(v) - 1, int(q * (len(v) - 1) + 0.5))]


def measure_workload(wl, alive, steps, warmup, with_failover=True):
    """Times tg_ew_forward on one resident workload: ``steps`` plain steps
    (host clock around the loop, one hipEvent after each step on the call's
    stream), a second pass through tg_ew_forward_timed for the per-stage
    means, the roofline of the dominant kernel (the gate/up GEMM), and, when
    the workload has a failure configuration, healthy and rerouted steps in
    interleaved blocks."""
    import torch

    from paper_2601_01310_amd import tg

    f = tg.EwForward(wl, alive)
    hip = HipEvents()
    stream = torch.cuda.current_stream()

    def timed_steps(n):
        evs = hip.create(n + 1)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        hip.record(evs[0], stream)
        for i in range(n):
            tg.tg_ew_forward(f.args, f.ws, f.ws_bytes, stream)
            hip.record(evs[i + 1], stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        per = sorted(hip.elapsed_ms(evs[i], evs[i + 1]) for i in range(n))
        hip.destroy(evs)
        return per, (t1 - t0) * 1e3 / n

    def stage_times(n):
        evs = hip.create(6 * n)
        torch.cuda.synchronize()
        for i in range(n):
            tg.tg_ew_forward_timed(f.args, f.ws, f.ws_bytes, evs[6 * i:6 * i + 6], stream)
        torch.cuda.synchronize()
        st = [sum(hip.elapsed_ms(evs[6 * i + j], evs[6 * i + j + 1]) for i in range(n)) / n
              for j in range(5)]
        hip.destroy(evs)
        return st

    for _ in range(warmup):
        f(stream)
    step_ev, ms = timed_steps(steps)
    stage_ms = stage_times(steps)
    P = int(f.slot_offsets[-1])
    counts = f.slot_counts.cpu()
    touched = int((counts > 0).sum())

    failover = None
    fail_alive = wl.alive_after_failure()
    if with_failover and not torch.equal(fail_alive, wl.alive):
        # Healthy and rerouted configurations alternate in blocks, so that
        # both see the same clock and temperature; p50 and the inter-quartile
        # range of each, and the cost with its own spread.
        n = max(steps, FAILOVER_BLOCK_STEPS)
        per = {"healthy": [], "failover": []}
        for _ in range(FAILOVER_BLOCKS // 2):
            for tag, al in (("healthy", wl.alive), ("failover", fail_alive)):
                f.set_alive(al)
                for _ in range(2):
                    f(stream)
                per[tag] += timed_steps(n)[0]
        f.set_alive(fail_alive)
        f(stream)
        torch.cuda.synchronize()
        fo_pairs = int(f.slot_offsets[-1])
        f.set_alive(alive)
        q = {t: (_pct(v, 0.25), _pct(v, 0.5), _pct(v, 0.75)) for t, v in per.items()}
        h, fo = q["healthy"], q["failover"]
        failover = {"step_ms_p50": fo[1], "step_ms_iqr": [fo[0], fo[2]],
                    "healthy_step_ms_p50": h[1], "healthy_step_ms_iqr": [h[0], h[2]],
                    "cost": fo[1] / h[1] - 1.0,
                    "cost_spread": (h[2] - h[0]) / h[1],
                    "routed_pairs": fo_pairs, "blocks": FAILOVER_BLOCKS, "steps_per_block": n}

    d, I = wl.d, wl.I
    roof = gateup_roofline(d, I, P, touched, stage_ms[2] * 1e-3)
    p50 = step_ev[len(step_ev) // 2]
    # Bytes the whole step must stream: every touched slot's three weight
    # matrices, the token rows and the outputs.
    step_bytes = touched * 3.0 * I * d * 2 + wl.T * d * 2.0 * 2
    return {"routed_pairs": P, "touched_slots": touched, "pairs_per_s": P / (ms * 1e-3),
            "ms_per_step": ms, "step_ms_p50": p50, "step_ms_mean": sum(step_ev) / len(step_ev),
            "stages_ms": dict(zip(STAGES, stage_ms)), "roofline": roof,
            "expert_ffn_tflops": 6.0 * d * I * P / ((stage_ms[2] + stage_ms[3]) * 1e-3) / 1e12,
            "step_flop_frac": 6.0 * d * I * P / (p50 * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "step_hbm_frac": step_bytes / (p50 * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "failover": failover}


def gateup_roofline(d, I, pairs, touched, seconds):
    """Roofline entry of the gate/up GEMM from its average launch time.

    Algorithmic flops 4·d·I per routed pair; algorithmic bytes the touched
    slots' W1/W3 (2·I·d bf16 each) plus the routed rows of x and h. At or
    above the ridge point (peak flops over peak bytes) the GEMM is reported
    against the bf16 MFMA peak, below it against HBM.
    """
    flop = 4.0 * d * I * pairs
    nbytes = touched * 2.0 * I * d * 2 + pairs * d * 2.0 + pairs * I * 2.0
    if flop / max(nbytes, 1.0) >= RIDGE_FLOP_PER_BYTE:
        achieved = flop / seconds / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS}
    else:
        achieved = nbytes / seconds / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS}
    return {"bound": roof["bound"], "kernel": "grouped_gemm gate/up + SwiGLU", **roof}


def compact(wl, r):
    """The summary of one extra workload carried in the benchmark line."""
    out = {"workload": f"T={wl.T} d={wl.d} E={wl.E} top-{wl.k} I={wl.I} slots={wl.S}",
           "routed_pairs": r["routed_pairs"], "touched_slots": r["touched_slots"],
           "pairs_per_s": r["pairs_per_s"], "step_ms_p50": r["step_ms_p50"],
           "ms_per_step": r["ms_per_step"],
           "stages_ms": {k: round(v, 4) for k, v in r["stages_ms"].items()},
           "roofline": dict(r["roofline"], traffic=measured_traffic(wl.name))}
    if r["roofline"]["bound"] == "hbm":
        out["step_hbm_frac"] = r["step_hbm_frac"]
    else:
        out["step_flop_frac"] = r["step_flop_frac"]
    if r["failover"] is not None:
        out["failover"] = r["failover"]
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mixtral")
    ap.add_argument("--failover", action="store_true",
                    help="time the run with the workload's failed primaries rerouted to shadows")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-failover", action="store_true",
                    help="skip the interleaved healthy / rerouted blocks (profiling runs)")
    ap.add_argument("--no-others", action="store_true",
                    help="time only the named workload (by default the mixtral line also carries "
                         "the DeepSeek-V3 share, skewed and decode workloads under 'workloads')")
    ap.add_argument("--knee", action="store_true",
                    help="expert FFN time against the expert batch size (prints one JSON line per "
                         "point instead of the benchmark line)")
    ap.add_argument("--shadow", action="store_true",
                    help="idle-shadow / concurrent-expert interference check (one JSON line)")
    ap.add_argument("--ckpt", action="store_true",
                    help="KV-segment checkpoint of one decode step: alone and alongside the "
                         "forward (one JSON line)")
    ap.add_argument("--partial", action="store_true",
                    help="partial-batch trigger + forward against the full forward (one JSON line)")
    ap.add_argument("--replay", action="store_true",
                    help="cost of replaying the failed primaries' pairs after a forward, against "
                         "the forward (one JSON line)")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the library references (bf16 GEMM, HBM read, copy) that the "
                         "roofline fraction is also reported against")
    ap.add_argument("--calib-copy", action="store_true",
                    help="first copy a 1 GiB device buffer 3 times (a plain copy of known size "
                         "that calibrates the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the expert-parallel "
              "exchange across GPUs is not implemented", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2601_01310_amd import synth, tg

    tg.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calib_copy:
        src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.knee:
        expert_batch_knee(dev)
        return
    if args.shadow:
        shadow_interference(dev)
        return
    wl = synth.make(args.workload, device=dev)
    if args.replay:
        replay_cost(wl, args.steps, args.warmup)
        return
    if args.partial:
        partial_batch_cost(wl, args.steps, args.warmup)
        return
    if args.ckpt:
        checkpoint_cost(wl, args.steps, args.warmup)
        return
    alive = wl.alive_after_failure() if args.failover else wl.alive
    res = measure_workload(wl, alive, args.steps, args.warmup,
                           with_failover=not (args.failover or args.no_failover))
    P, touched, stage_ms = res["routed_pairs"], res["touched_slots"], res["stages_ms"]
    d, I = wl.d, wl.I
    line = {
        "metric": "routed token-expert pairs/sec for EW forward",
        "value": res["pairs_per_s"],
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: T={wl.T} d={d} E={wl.E} top-{wl.k} I={I} "
                               f"slots={wl.S}" + (" failover" if args.failover else ""),
                   "routed_pairs": P, "touched_slots": touched},
        "roofline": dict(res["roofline"], traffic=measured_traffic(args.workload)),
        "step_ms_p50": res["step_ms_p50"],
        "step_ms_mean": res["step_ms_mean"],
        "stages_ms": stage_ms,
        "expert_ffn_tflops": res["expert_ffn_tflops"],
    }
    if res.get("failover") is not None:
        line["failover"] = res["failover"]
    if not args.no_others and args.workload == "mixtral" and not args.failover:
        # The other full-size workloads, each timed the same way (compact).
        line["workloads"] = {}
        for name in OTHER_WORKLOADS:
            wl2 = synth.make(name, device=dev)
            r2 = measure_workload(wl2, wl2.alive, max(args.steps, 20), args.warmup,
                                  with_failover=True)
            line["workloads"][name] = compact(wl2, r2)
            del wl2
            torch.cuda.empty_cache()
    if not args.no_peaks:
        mp = measured_peaks(dev)
        roof = line["roofline"]
        ref = (mp["bf16_gemm_tflops"] if roof["bound"] == "mfma"
               else max(mp["hbm_read_tbps"], mp["hbm_copy_tbps"]) * 1e3)
        line["measured_peaks"] = mp
        line["roofline"]["frac_of_measured"] = roof["achieved"] / ref
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
