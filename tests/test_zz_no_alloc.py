"""tg_ew_forward_noalloc: the forward on the library's own scratch area.

The entry point must compute exactly what tg_ew_forward computes on a caller
workspace (same kernels), including on a second call with a smaller batch
that finds the first call's contents still in the scratch area, and must
reject a batch too large for the area before enqueuing anything.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2601_01310_amd import synth, tg
from tests._util import host, u16

DEV = "cuda"
P = 0x1000  # bogus non-NULL address: the calls below that use it fail validation first


def _args(wl, out, **outs):
    return tg.make_ew_args(wl.T, wl.d, wl.E, wl.k, wl.I, wl.S, wl.R, wl.x, wl.wg, wl.logits,
                           wl.ert, wl.alive, wl.w13, wl.w2, out, **outs)


def _outputs(wl):
    dev = wl.x.device
    T, k, S = wl.T, wl.k, wl.S
    return dict(topk_ids=torch.empty((T, k), dtype=torch.int32, device=dev),
                topk_w=torch.empty((T, k), dtype=torch.float32, device=dev),
                pair_slot=torch.empty((T, k), dtype=torch.int32, device=dev),
                slot_counts=torch.empty((S,), dtype=torch.int32, device=dev),
                slot_offsets=torch.empty((S + 1,), dtype=torch.int32, device=dev),
                pair_row=torch.empty((T, k), dtype=torch.int32, device=dev),
                n_unserved=torch.empty((1,), dtype=torch.int32, device=dev))


def _run(wl, noalloc):
    out = torch.full((wl.T, wl.d), 3, dtype=torch.int16, device=wl.x.device).view(torch.bfloat16)
    o = _outputs(wl)
    a = _args(wl, out, **o)
    if noalloc:
        assert tg.tg_ew_forward_workspace(a) <= tg.NOALLOC_SCRATCH_BYTES
        tg.tg_ew_forward_noalloc(a)
    else:
        wsb = tg.tg_ew_forward_workspace(a)
        tg.tg_ew_forward(a, tg.workspace(wsb, wl.x.device), wsb)
    torch.cuda.synchronize()
    res = {k_: host(v) for k_, v in o.items()}
    res["out"] = u16(out)
    return res


@pytest.mark.gpu
def test_noalloc_forward_equals_the_workspace_forward_on_two_calls_in_a_row():
    """A DeepSeek-V3-shaped decode batch (logits mode, 256 experts, 40 slots)
    and then a smaller Mixtral-like batch (weights mode, another layout of
    the same scratch area): every output bit-identical to tg_ew_forward on a
    caller workspace, each call after the other."""
    big = synth.make("dsv3_decode", device=DEV, T=300)
    small = synth.make_custom(T=77, d=512, E=8, k=2, I=384, n_local=8, shadow_experts=[0, 5],
                              gate="weights", seed=31, device=DEV)
    for wl in (big, small):
        print(f"[gpu] noalloc {wl.name} T={wl.T} d={wl.d} E={wl.E}", flush=True)
        got = _run(wl, noalloc=True)
        ref = _run(wl, noalloc=False)
        assert int(got["slot_offsets"][-1]) > 0
        for key in ref:
            assert np.array_equal(got[key], ref[key]), f"{wl.name}: {key} differs"
    # a second round in the reverse order, with dead slots: the scratch area
    # now holds the small batch's intermediates
    alive = big.alive.clone()
    alive[torch.tensor([0, 5, 33], device=DEV)] = 0
    big.alive = alive
    got, ref = _run(big, noalloc=True), _run(big, noalloc=False)
    for key in ref:
        assert np.array_equal(got[key], ref[key]), f"dead slots: {key} differs"


def test_noalloc_forward_rejects_a_batch_beyond_its_scratch_area():
    """Checked on the host before any HIP call (runs without a GPU)."""
    lib = tg.load()
    a = tg.EwArgs()
    a.T, a.d, a.E, a.k, a.I, a.S, a.R = 4096, 7168, 256, 8, 2048, 40, 2
    for n in ("x", "logits_in", "ert", "slot_alive", "w13", "w2", "out"):
        setattr(a, n, P)
    assert lib.tg_ew_forward_workspace(ctypes.byref(a)) > tg.NOALLOC_SCRATCH_BYTES
    assert lib.tg_ew_forward_noalloc(ctypes.byref(a), None) == tg.TG_ERR_WORKSPACE
    assert b"scratch area holds 67108864" in lib.tg_last_error()
    a.T = 0
    a.k = 300  # invalid arguments are reported as by tg_ew_forward
    assert lib.tg_ew_forward_noalloc(ctypes.byref(a), None) == tg.TG_ERR_BAD_DIM
    assert lib.tg_ew_forward_noalloc(None, None) == tg.TG_ERR_NULL_ARG


def test_decode_batch_limit_stated_in_the_header():
    """The header states that the scratch area covers a decode step of 432
    tokens at DeepSeek-V3 expert shapes (d = 7168, I = 2048, 256 experts,
    top-8, 40 slots)."""
    lib = tg.load()
    a = tg.EwArgs()
    a.d, a.E, a.k, a.I, a.S, a.R = 7168, 256, 8, 2048, 40, 2
    for n in ("x", "logits_in", "ert", "slot_alive", "w13", "w2", "out"):
        setattr(a, n, P)
    a.T = 432
    assert lib.tg_ew_forward_workspace(ctypes.byref(a)) <= tg.NOALLOC_SCRATCH_BYTES
    a.T = 460
    assert lib.tg_ew_forward_workspace(ctypes.byref(a)) > tg.NOALLOC_SCRATCH_BYTES
