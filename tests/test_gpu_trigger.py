"""EW-side partial-batch trigger (§5.2) on the GPU: its decision and batch
mask against the oracle's definition, a wait that ends when the host
delivers, and a trigger followed by the forward on the partial batch.

Every trigger call here ends by itself: the flags are set before the launch
or by the host during the wait, and every call has a poll budget.
"""
import time

import numpy as np
import pytest
import torch

from oracle import moe_ew as O
from paper_2601_01310_amd import synth, tg
from tests import _gpu as G
from tests._util import host, u16

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _trigger(delivered, alive, chunk_rows, T, min_rows, spin_limit):
    A = len(alive)
    tv = torch.full((max(T, 1),), 7, dtype=torch.uint8, device=DEV)
    st = torch.full((4,), -1, dtype=torch.int32, device=DEV)
    d = torch.tensor(delivered, dtype=torch.int32, device=DEV)
    tg.tg_batch_trigger(d, torch.tensor(alive, dtype=torch.uint8, device=DEV),
                        torch.tensor(chunk_rows, dtype=torch.int32, device=DEV), A, T, min_rows,
                        spin_limit, tv, st)
    torch.cuda.synchronize()
    return host(tv)[:T], host(st)


def test_trigger_decisions_match_the_oracle():
    rng = np.random.default_rng(12)
    for case in range(60):
        A = int(rng.integers(1, 9))
        sizes = rng.integers(0, 40, size=A)
        chunk_rows = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
        T = int(chunk_rows[-1]) + int(rng.integers(0, 5)) - int(rng.integers(0, 3))
        T = max(T, 0)
        delivered = (rng.random(A) < 0.7).astype(np.int32).tolist()
        alive = (rng.random(A) < 0.85).astype(np.uint8).tolist()
        min_rows = int(rng.integers(0, max(T, 1) + 10))
        cond, tv_o, rows_o, n_o = O.batch_trigger(delivered, alive, chunk_rows.tolist(), T, min_rows)
        tv, st = _trigger(delivered, alive, chunk_rows.tolist(), T, min_rows, spin_limit=3)
        assert np.array_equal(tv, tv_o), case
        assert st.tolist() == [cond, rows_o, n_o, 3 if cond == 2 else 1], case


def test_trigger_waits_until_the_host_delivers():
    """Flags in pinned host memory, all zero at launch; the host sets them
    while the kernel waits (budget of ~2 s of polls)."""
    A, T = 4, 64
    flags = torch.zeros(A, dtype=torch.int32, pin_memory=True)
    alive = torch.tensor([1, 1, 0, 1], dtype=torch.uint8, device=DEV)
    chunk_rows = torch.tensor([0, 16, 32, 48, 64], dtype=torch.int32, device=DEV)
    tv = torch.zeros(T, dtype=torch.uint8, device=DEV)
    st = torch.zeros(4, dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()
    tg.tg_batch_trigger(flags, alive, chunk_rows, A, T, T, 500_000, tv, st)
    time.sleep(0.05)
    flags.numpy()[[0, 1, 3]] = 1
    torch.cuda.synchronize()
    s = host(st).tolist()
    assert s[0] == 0 and s[1] == 48 and s[2] == 3 and s[3] > 1, s
    assert host(tv).tolist() == [1] * 32 + [0] * 16 + [1] * 16


def test_trigger_then_forward_on_the_partial_batch():
    """Four AWs deliver the tiny workload's 64 tokens in chunks of 16; AW 2
    never delivers and the trigger fires on the minimum batch; the forward
    then computes exactly the other AWs' tokens."""
    wl = synth.make("tiny", device=DEV)
    A = 4
    chunk_rows = torch.tensor([0, 16, 32, 48, 64], dtype=torch.int32, device=DEV)
    delivered = torch.tensor([1, 1, 0, 1], dtype=torch.int32, device=DEV)
    alive = torch.ones(A, dtype=torch.uint8, device=DEV)
    tv = torch.empty(wl.T, dtype=torch.uint8, device=DEV)
    st = torch.empty(4, dtype=torch.int32, device=DEV)
    f = tg.EwForward(wl, token_valid=tv)
    tg.tg_batch_trigger(delivered, alive, chunk_rows, A, wl.T, 40, 1000, tv, st)
    f()
    torch.cuda.synchronize()
    assert host(st).tolist()[:3] == [1, 48, 3]
    keep = host(tv).astype(bool)
    assert keep.tolist() == [True] * 32 + [False] * 16 + [True] * 16
    a = dict(x=host(wl.x), wg=host(wl.wg), logits=None, k=wl.k, ert=host(wl.ert),
             alive=host(wl.alive))
    r = O.ew_forward(**a, w13=u16(wl.w13), w2=u16(wl.w2), token_valid=keep.astype(np.uint8))
    assert np.array_equal(host(f.pair_slot), r["pair_slot"])
    G.assert_close_bf16(u16(f.out), r["out"], "out after trigger")
    assert not u16(f.out)[~keep].any()
