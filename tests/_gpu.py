"""Drivers shared by the GPU tests: run the HIP path through the C ABI, run
the oracle on the same inputs, and compare (no method arithmetic here)."""
from __future__ import annotations

import numpy as np
import torch

from oracle import moe_ew as O
from paper_2601_01310_amd import synth, tg
from tests._util import bf16_bits_to_f32, host, u16, within_tol

ATOL, RTOL = 2e-2, 1e-2      # bf16 outputs, float32 accumulation
W_ATOL = 1e-6                # float32 gate weights vs float64


def np_inputs(wl, alive=None):
    return dict(x=host(wl.x), wg=None if wl.wg is None else host(wl.wg),
                logits=None if wl.logits is None else host(wl.logits), k=wl.k,
                ert=host(wl.ert), alive=host(wl.alive if alive is None else alive))


def run_stepwise(wl, alive=None):
    """Each entry point called on its own, in order; returns host copies of
    every intermediate."""
    dev = wl.x.device
    alive = wl.alive if alive is None else alive
    T, k, S, d, I, E = wl.T, wl.k, wl.S, wl.d, wl.I, wl.E
    ids = torch.empty((T, k), dtype=torch.int32, device=dev)
    w = torch.empty((T, k), dtype=torch.float32, device=dev)
    logits = torch.empty((T, E), dtype=torch.float32, device=dev) if wl.wg is not None else None
    tg.tg_gate_topk(wl.x if wl.wg is not None else None, wl.wg, wl.logits, T, d, E, k, logits,
                    ids, w)
    pair_slot = torch.empty((T, k), dtype=torch.int32, device=dev)
    counts = torch.empty((S,), dtype=torch.int32, device=dev)
    offsets = torch.empty((S + 1,), dtype=torch.int32, device=dev)
    perm = torch.full((max(T * k, 1),), -7, dtype=torch.int32, device=dev)
    pair_row = torch.empty((T, k), dtype=torch.int32, device=dev)
    x_perm = torch.empty((max(T * k, 1), d), dtype=torch.bfloat16, device=dev)
    nu = torch.empty((1,), dtype=torch.int32, device=dev)
    wsb = tg.tg_remap_dispatch_workspace(T, k, S)
    ws = tg.workspace(wsb, dev)
    tg.tg_remap_dispatch(ids, T, k, wl.ert, E, wl.R, alive, S, wl.x, d, pair_slot, counts, offsets,
                         perm, pair_row, x_perm, nu, ws, wsb)
    h = torch.empty((max(T * k, 1), I), dtype=torch.bfloat16, device=dev)
    y = torch.empty((max(T * k, 1), d), dtype=torch.bfloat16, device=dev)
    tg.tg_expert_ffn_grouped(x_perm, offsets, S, T * k, wl.w13, wl.w2, d, I, h, y)
    out = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    tg.tg_combine(y, pair_row, w, T, k, d, out)
    torch.cuda.synchronize()
    P = int(offsets[-1])
    return dict(logits=None if logits is None else host(logits), ids=host(ids), w=host(w),
                pair_slot=host(pair_slot), counts=host(counts), offsets=host(offsets),
                perm=host(perm)[:P], pair_row=host(pair_row), n_unserved=int(nu[0]),
                x_perm=u16(x_perm[:P]), h=u16(h[:P]), y=u16(y[:P]), out=u16(out))


def run_fused(wl, alive=None):
    """tg_ew_forward; returns host copies of its outputs."""
    f = tg.EwForward(wl, alive)
    f()
    torch.cuda.synchronize()
    return dict(ids=host(f.topk_ids), w=host(f.topk_w), pair_slot=host(f.pair_slot),
                counts=host(f.slot_counts), offsets=host(f.slot_offsets),
                pair_row=host(f.pair_row), n_unserved=int(f.n_unserved[0]), out=u16(f.out))


def assert_routing_equal(g, r, *, check_perm=True):
    assert np.array_equal(g["ids"], r["ids"]), "topk ids differ"
    assert np.abs(g["w"].astype(np.float64) - r["w"]).max() <= W_ATOL, "gate weights differ"
    assert np.array_equal(g["pair_slot"], r["pair_slot"]), "pair_slot differs"
    assert g["n_unserved"] == r["n_unserved"], (g["n_unserved"], r["n_unserved"])
    assert np.array_equal(g["counts"], r["counts"]), "slot counts differ"
    assert np.array_equal(g["offsets"], r["offsets"]), "slot offsets differ"
    assert np.array_equal(g["pair_row"], r["pair_row"]), "pair_row differs"
    if check_perm:
        assert np.array_equal(g["perm"], r["perm"]), "perm differs"


def assert_close_bf16(g, r, what):
    ok, max_abs, worst = within_tol(g, r, ATOL, RTOL)
    assert ok, f"{what}: max |err| {max_abs} at flat index {worst}"


def out_term_scale(r):
    """sum_j |w[t,j] * y[pair_row[t,j], c]| for every output element, from
    an oracle result (the size of the terms that the combine sums)."""
    T, k = r["pair_row"].shape
    yf = bf16_bits_to_f32(r["y"]).astype(np.float64) if len(r["y"]) else None
    scale = np.zeros((T, r["out"].shape[1]), np.float64)
    for j in range(k):
        rows = r["pair_row"][:, j]
        m = rows >= 0
        if m.any():
            scale[m] += np.abs(r["w"][m, j])[:, None] * np.abs(yf[rows[m]])
    return scale


def assert_out_close(g_out, r, what):
    """A forward's out against the oracle's, every element.

    out is the gate-weighted sum of the per-pair outputs y, each rounded to
    bf16. The kernel's y (float32 accumulation) and the oracle's (float64)
    can round to neighbouring bf16 values: a difference of up to one bf16
    ulp of |y|, at most 2^-7 |y|, that reaches out undiminished when the
    token's terms cancel. The relative part of the 2e-2 / 1e-2 tolerance is
    therefore taken against the size of the summed terms,
    sum_j |w_j y_j| >= |out|: |gpu - ref| <= atol + rtol * sum_j |w_j y_j|.
    Returns the number of elements outside the plain elementwise bound (the
    cancellation cases), for the record."""
    g = bf16_bits_to_f32(g_out).astype(np.float64)
    ref = bf16_bits_to_f32(r["out"]).astype(np.float64)
    err = np.abs(g - ref)
    scale = np.maximum(out_term_scale(r), np.abs(ref))
    bad = err > ATOL + RTOL * scale
    if bad.any():
        i = int(np.argmax(err - (ATOL + RTOL * scale)))
        raise AssertionError(f"{what}: |err| {err.flat[i]} at flat index {i}, |ref| "
                             f"{abs(ref.flat[i])}, sum of |terms| {scale.flat[i]}")
    return int((err > ATOL + RTOL * np.abs(ref)).sum())


def sample_tokens(route, T, n, seed):
    """A seeded sample of tokens, plus tokens with no local pair and tokens
    with the most local pairs (when present)."""
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(T, size=min(n, T), replace=False).tolist())
    nloc = (route["pair_slot"] >= 0).sum(axis=1)
    for cand in (np.flatnonzero(nloc == 0)[:2], np.argsort(-nloc, kind="stable")[:2]):
        pick.update(int(c) for c in cand)
    return sorted(pick)


def oracle_sampled_out(wl, alive, tokens):
    a = np_inputs(wl, alive)
    return O.ew_forward_tokens(tokens, a["x"], a["wg"], a["logits"], a["k"], a["ert"], a["alive"],
                               lambda s: u16(wl.w13[s]), lambda s: u16(wl.w2[s]))
