"""Token rows too large to be read in place: the permuted-copy path.

The gate/up GEMM reads each routed pair's token row straight from x through
the permutation when x is addressable with 32-bit byte offsets. With
2*T*d >= 2^31 bytes the forward and the replay instead gather the rows into
a permuted copy first and run the GEMM on that copy. Here x is exactly
2 GiB (T = 262144 tokens of d = 4096), and every token's output is checked
against the oracle (computed slot by slot and in chunks of tokens: each row
of the expert FFN and each token's combine depend only on their own inputs).
"""
import numpy as np
import pytest
import torch

from oracle import moe_ew as O
from paper_2601_01310_amd import synth, tg
from tests import _gpu as G
from tests._util import host, u16

pytestmark = pytest.mark.gpu
DEV = "cuda"
T, D = 262144, 4096


@pytest.fixture(scope="module")
def big():
    print(f"[gpu] large x: T={T} d={D} ({2 * T * D} bytes)", flush=True)
    wl = synth.make_custom(T=T, d=D, E=8, k=1, I=128, n_local=8, shadow_experts=[0, 5],
                           gate="weights", seed=41, device=DEV, fail_experts=[5])
    assert 2 * wl.T * wl.d >= 1 << 31
    x, wg, ert, alive = host(wl.x), host(wl.wg), host(wl.ert), host(wl.alive)
    w13, w2 = u16(wl.w13), u16(wl.w2)
    r = O.route(x, wg, None, wl.k, ert, alive)
    P = int(r["offsets"][-1])
    y = np.zeros((P, D), np.uint16)
    for s in range(wl.S):
        a, b = int(r["offsets"][s]), int(r["offsets"][s + 1])
        if b > a:
            y[a:b] = O.expert_ffn(x[r["perm"][a:b] // wl.k], w13[s], w2[s])[1]
    r.update(y=y, out=_combine_chunked(y, r["pair_row"], r["w"]))
    print(f"[gpu] large x: oracle done, P={P}", flush=True)
    return wl, r


def _combine_chunked(y, pair_row, w, chunk=16384):
    """The oracle's combine, a chunk of tokens at a time (each token's sum
    reads only its own rows of y)."""
    outs = []
    for t0 in range(0, len(pair_row), chunk):
        pr = pair_row[t0:t0 + chunk]
        rows = pr[pr >= 0]
        sub = np.full_like(pr, -1)
        sub[pr >= 0] = np.arange(rows.size, dtype=np.int32)
        outs.append(O.combine(y[rows], sub, w[t0:t0 + chunk]))
    return np.concatenate(outs)


def _g(f):
    return dict(ids=host(f.topk_ids), w=host(f.topk_w), pair_slot=host(f.pair_slot),
                counts=host(f.slot_counts), offsets=host(f.slot_offsets),
                pair_row=host(f.pair_row), n_unserved=int(f.n_unserved[0]), out=u16(f.out))


def test_forward_with_permuted_copy_matches_oracle(big):
    wl, r = big
    f = tg.EwForward(wl, keep_y=True)
    f()
    torch.cuda.synchronize()
    g = _g(f)
    P = int(g["offsets"][-1])
    G.assert_routing_equal(g, r, check_perm=False)
    G.assert_close_bf16(u16(f.y[:P]), r["y"], "y (every row)")
    G.assert_close_bf16(g["out"], _combine_chunked(u16(f.y[:P]), g["pair_row"],
                                                   g["w"].astype(np.float64)),
                        "out vs the oracle's combine of the kernel's y")
    G.assert_out_close(g["out"], r, "out (every token)")
    # failed primary rerouted to its shadow: bit-identical output
    fo = tg.EwForward(wl, wl.alive_after_failure())
    fo()
    torch.cuda.synchronize()
    assert np.array_equal(u16(fo.out), g["out"]), "failover output differs"


def test_replay_with_permuted_copy_matches_oracle(big):
    """Expert 5's primary fails after the forward and its outputs are lost
    (NaN): its pairs are gathered into a permuted copy, recomputed on the
    shadow and merged; the output equals the forward under the new mask bit
    for bit, and the oracle."""
    wl, r = big
    f = tg.EwForward(wl, keep_y=True)
    f()
    alive1 = wl.alive_after_failure()
    # the failed slot's per-pair outputs and its tokens' out rows never arrived
    hit = f.pair_slot == int(wl.ert[5, 0])
    f.y[f.pair_row[hit].long()] = float("nan")
    f.out[hit.any(dim=1)] = float("nan")
    replay_slot, n_rep, _ = f.replay(alive1)
    torch.cuda.synchronize()
    assert int(n_rep[0]) == int(r["counts"][5]) > 0
    rs = host(replay_slot)
    assert np.array_equal(rs >= 0, r["pair_slot"] == 5)
    assert (rs[rs >= 0] == wl.S - 1).all()  # expert 5's shadow is the last slot
    out_replayed = u16(f.out)
    del f
    fo = tg.EwForward(wl, alive1)
    fo()
    torch.cuda.synchronize()
    assert np.array_equal(out_replayed, u16(fo.out)), "replay differs from the failover forward"
    G.assert_out_close(out_replayed, r, "out after replay (every token)")
