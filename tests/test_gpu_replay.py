"""Replay of failed pairs (§5.1) and the EW-side partial batch (§5.2) on the
HIP path, against the oracle and against the plain forward.

Replay: a forward runs with every slot alive; then slots fail before its
result is used, the failed slots' per-pair outputs (and the out rows of
their tokens) are overwritten with NaN as if they had never arrived, and
tg_ew_replay must restore exactly what a forward with the new mask gives
(bit for bit, shadows hold byte copies of their primaries' weights).

Partial batch: tokens outside the batch are not routed and get +0; the
others' results are bit-identical to a forward over them alone.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import moe_ew as O
from paper_2601_01310_amd import synth, tg
from tests import _gpu as G
from tests._util import host, u16

pytestmark = pytest.mark.gpu
DEV = "cuda"
NAN_BF16 = float("nan")


def _lose_outputs(f, dead):
    """NaN into the per-pair outputs of the pairs on the slots in ``dead``
    and into the out rows of their tokens."""
    hit = torch.zeros_like(f.pair_slot, dtype=torch.bool)
    for s in dead:
        hit |= f.pair_slot == s
    rows = f.pair_row[hit].long()
    f.y[rows] = NAN_BF16
    f.out[hit.any(dim=1)] = NAN_BF16


def _replay_case(wl, alive1, dead, token_valid=None, oracle=True):
    """First pass with every slot alive, lose the outputs of ``dead``, replay
    under ``alive1``; compare with a forward under ``alive1``."""
    f = tg.EwForward(wl, keep_y=True, token_valid=token_valid)
    f()
    torch.cuda.synchronize()
    first = dict(ids=host(f.topk_ids), w=host(f.topk_w).astype(np.float64),
                 pair_slot=host(f.pair_slot), pair_row=host(f.pair_row),
                 y=u16(f.y), out=u16(f.out))
    _lose_outputs(f, dead)
    replay_slot, n_rep, n_un = f.replay(alive1)
    torch.cuda.synchronize()
    got = u16(f.out)
    ref = tg.EwForward(wl, alive1, token_valid=token_valid)
    ref()
    torch.cuda.synchronize()
    assert np.array_equal(got, u16(ref.out)), "replayed output differs from the failover forward"
    assert int(n_un[0]) == int(ref.n_unserved[0])
    if oracle:
        # The oracle's replay on the GPU first pass's routing and outputs.
        a = G.np_inputs(wl, alive1)
        out_o, rs, nr, nu = O.replay(a["x"], wl.k, a["ert"], a["alive"], u16(wl.w13),
                                     u16(wl.w2), first["ids"], first["w"], first["pair_slot"],
                                     first["pair_row"], first["y"], first["out"])
        assert np.array_equal(host(replay_slot), rs)
        assert int(n_rep[0]) == nr and int(n_un[0]) == nu
        G.assert_close_bf16(got, out_o, "replayed out vs oracle replay")
    return f, ref, int(n_rep[0])


@pytest.fixture(scope="module")
def tiny():
    print("[gpu] replay tiny", flush=True)
    return synth.make("tiny", device=DEV)


def test_replay_after_failure_matches_failover_forward_and_oracle(tiny):
    alive1 = tiny.alive_after_failure()
    f, ref, n = _replay_case(tiny, alive1, dead=[3])
    assert n == int((f.pair_slot == 3).sum()) > 0
    r = O.ew_forward(**G.np_inputs(tiny, alive1), w13=u16(tiny.w13), w2=u16(tiny.w2))
    G.assert_close_bf16(u16(f.out), r["out"], "replayed out")


def test_replay_drops_pairs_of_an_expert_without_live_candidates(tiny):
    alive1 = tiny.alive.clone()
    alive1[1] = 0
    _, _, n = _replay_case(tiny, alive1, dead=[1])
    assert n == 0


def test_replay_with_nothing_failed_is_a_no_op(tiny):
    f = tg.EwForward(tiny, keep_y=True)
    f()
    before = u16(f.out)
    rs, n_rep, n_un = f.replay(tiny.alive)
    torch.cuda.synchronize()
    assert np.array_equal(u16(f.out), before)
    assert (host(rs) == -1).all() and int(n_rep[0]) == 0 and int(n_un[0]) == 0


def test_replay_computes_pairs_that_were_unserved(tiny):
    alive0 = tiny.alive.clone()
    alive0[3] = 0
    alive0[9] = 0
    f = tg.EwForward(tiny, alive0, keep_y=True)
    f()
    n_first = int(f.n_unserved[0])
    rs, n_rep, n_un = f.replay(tiny.alive)
    ref = tg.EwForward(tiny)
    ref()
    torch.cuda.synchronize()
    assert np.array_equal(u16(f.out), u16(ref.out))
    assert int(n_rep[0]) == n_first > 0 and int(n_un[0]) == 0
    assert (host(rs)[host(f.topk_ids) == 3] == 3).all()


def test_replay_repeated_on_successive_failures(tiny):
    """Two failures, two replays: each replay starts from the state the last
    one left (its pair_slot is the first pass's, so the second replay also
    recomputes the first one's pairs; the output is still the forward's)."""
    f = tg.EwForward(tiny, keep_y=True)
    f()
    a1 = tiny.alive_after_failure()
    f.replay(a1)
    a2 = a1.clone()
    a2[0] = 0  # expert 0's primary too; slot 8 is its shadow
    f.replay(a2)
    ref = tg.EwForward(tiny, a2)
    ref()
    torch.cuda.synchronize()
    assert np.array_equal(u16(f.out), u16(ref.out))


REPLAY_CASES = [
    # T, d, E, k, I, n_local, shadows, gate, seed
    (37, 512, 16, 4, 384, 12, [1, 5, 11], "weights", 202),
    (200, 256, 64, 6, 256, 20, [0, 7], "logits", 203),
    (300, 768, 256, 8, 128, 32, [3, 4, 30], "logits", 205),
    (1000, 256, 4, 4, 128, 4, [2, 2], "weights", 207),
    (1024, 256, 32, 4, 128, 24, [0, 3], "logits", 208),  # 4096 pairs: the one-block dispatch's limit
    (700, 256, 1024, 8, 128, 1000, [3, 77], "logits", 209),  # 1002 slots x 22 chunks: separate scan
]


@pytest.mark.parametrize("case", REPLAY_CASES, ids=[f"T{c[0]}_E{c[2]}_k{c[3]}" for c in REPLAY_CASES])
def test_replay_random_shapes(case):
    T, d, E, k, I, n_local, shadows, gate, seed = case
    print(f"[gpu] replay case {case}", flush=True)
    wl = synth.make_custom(T=T, d=d, E=E, k=k, I=I, n_local=n_local, shadow_experts=shadows,
                           gate=gate, seed=seed, device=DEV)
    rng = np.random.default_rng(seed)
    dead = rng.choice(wl.S, size=max(1, wl.S // 4), replace=False).tolist()
    alive1 = wl.alive.clone()
    alive1[torch.tensor(dead, device=DEV)] = 0
    _replay_case(wl, alive1, dead)


@pytest.mark.parametrize("name", ["mixtral", "dsv3_skew"])
def test_replay_full_size(name):
    """The workload's failure configuration (mixtral: expert 5's primary;
    skewed DeepSeek share: the 4 hottest primaries) happens after the first
    pass; the replay must give the failover forward's output bit for bit."""
    print(f"[gpu] replay full-size {name}", flush=True)
    wl = synth.make(name, device=DEV)
    alive1 = wl.alive_after_failure()
    dead = torch.nonzero((wl.alive == 1) & (alive1 == 0)).flatten().tolist()
    f, _, n = _replay_case(wl, alive1, dead, oracle=False)
    assert n == int(sum(int((f.pair_slot == s).sum()) for s in dead)) > 0


# ---------------------------------------------------------------- partial batch (§5.2)


@pytest.mark.parametrize("name", ["tiny", "dsv3_decode"])
def test_partial_batch_matches_forward_on_the_included_tokens(name):
    print(f"[gpu] partial batch {name}", flush=True)
    wl = synth.make(name, device=DEV)
    valid = (torch.rand(wl.T, generator=torch.Generator().manual_seed(4)) < 0.6).to(torch.uint8)
    f = tg.EwForward(wl, token_valid=valid.to(DEV))
    f()
    keep = valid.bool()
    kd = keep.to(DEV)
    sub = dataclasses.replace(wl, T=int(keep.sum()), x=wl.x[kd].contiguous(),
                              logits=None if wl.logits is None else wl.logits[kd].contiguous())
    g = tg.EwForward(sub)
    g()
    torch.cuda.synchronize()
    out = u16(f.out)
    assert np.array_equal(out[keep.numpy()], u16(g.out))
    assert not out[~keep.numpy()].any()
    ps = host(f.pair_slot)
    assert (ps[~keep.numpy()] == -2).all() and (host(f.pair_row)[~keep.numpy()] == -1).all()
    assert np.array_equal(ps[keep.numpy()], host(g.pair_slot))
    assert int(f.n_unserved[0]) == int(g.n_unserved[0])
    if name == "tiny":
        a = G.np_inputs(wl)
        r = O.ew_forward(**a, w13=u16(wl.w13), w2=u16(wl.w2), token_valid=valid.numpy())
        assert np.array_equal(ps, r["pair_slot"])
        G.assert_close_bf16(out, r["out"], "partial-batch out")


def test_replay_within_a_partial_batch(tiny):
    valid = (torch.rand(tiny.T, generator=torch.Generator().manual_seed(8)) < 0.5).to(torch.uint8)
    f, _, _ = _replay_case(tiny, tiny.alive_after_failure(), dead=[3], token_valid=valid.to(DEV))
    assert not u16(f.out)[~valid.bool().numpy()].any()
