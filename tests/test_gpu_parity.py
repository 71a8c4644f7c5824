"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Integer results (top-k ids, slots, counts, offsets, permutation, rows) must
match bit for bit; bf16 results within |gpu - ref| <= 2e-2 + 1e-2 |ref|;
gate weights within 1e-6. A run with failed primaries rerouted to shadow
slots must reproduce the no-failure output bit for bit (§5.1, §5.3).
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


def _oracle_full(wl, alive=None):
    a = G.np_inputs(wl, alive)
    return O.ew_forward(**a, w13=u16(wl.w13), w2=u16(wl.w2))


@pytest.fixture(scope="module")
def tiny():
    print("[gpu] tiny workload", flush=True)
    return synth.make("tiny", device=DEV)


def test_tiny_each_entry_point_matches_oracle(tiny):
    g = G.run_stepwise(tiny)
    r = _oracle_full(tiny)
    assert np.array_equal(g["logits"], r["logits"]), "float32 logits differ"
    G.assert_routing_equal(g, r)
    assert np.array_equal(g["x_perm"], r["x_perm"])
    G.assert_close_bf16(g["h"], r["h"], "h")
    G.assert_close_bf16(g["y"], r["y"], "y")
    G.assert_close_bf16(g["out"], r["out"], "out")


def test_tiny_fused_matches_stepwise_and_oracle(tiny):
    f = G.run_fused(tiny)
    s = G.run_stepwise(tiny)
    r = _oracle_full(tiny)
    G.assert_routing_equal(f, r, check_perm=False)
    assert np.array_equal(f["out"], s["out"]), "fused and stepwise outputs differ"
    G.assert_close_bf16(f["out"], r["out"], "out")


def test_tiny_failure_rerouted_to_shadow_is_bit_identical(tiny):
    base = G.run_fused(tiny)
    alive = tiny.alive_after_failure()  # expert 3's primary fails
    fail = G.run_fused(tiny, alive)
    r = _oracle_full(tiny, alive)
    G.assert_routing_equal(fail, r, check_perm=False)
    assert fail["counts"][3] == 0 and fail["counts"][9] == base["counts"][3]
    assert np.array_equal(fail["out"], base["out"])


def test_combine_entry_point_on_oracle_intermediates(tiny):
    r = _oracle_full(tiny)
    P = int(r["offsets"][-1])
    y = torch.from_numpy(r["y"].view(np.int16)).view(torch.bfloat16).to(DEV)
    pr = torch.from_numpy(r["pair_row"]).to(DEV)
    w = torch.from_numpy(r["w"].astype(np.float32)).to(DEV)
    out = torch.empty((tiny.T, tiny.d), dtype=torch.bfloat16, device=DEV)
    tg.tg_combine(y, pr, w, tiny.T, tiny.k, tiny.d, out)
    torch.cuda.synchronize()
    assert P == y.shape[0]
    G.assert_close_bf16(u16(out), r["out"], "combine")


def test_ffn_entry_point_rows_independent_of_position(tiny):
    """The same rows placed at different offsets and in different slots with
    equal weights give identical bits."""
    d, I = tiny.d, tiny.I
    rows = tiny.x[:40].contiguous()
    x_perm = torch.cat([rows[:13], rows, rows[13:]]).contiguous()  # 13 | 40 | 27 rows
    # slot 0 gets 13 rows, slot 3 gets 40 rows, slot 9 (shadow of expert 3) 27
    offsets = torch.zeros(tiny.S + 1, dtype=torch.int32)
    cnt = torch.zeros(tiny.S, dtype=torch.int32)
    cnt[0], cnt[3], cnt[9] = 13, 40, 27
    offsets[1:] = torch.cumsum(cnt, 0)
    offsets = offsets.to(DEV)
    h = torch.empty((80, I), dtype=torch.bfloat16, device=DEV)
    y = torch.empty((80, d), dtype=torch.bfloat16, device=DEV)
    tg.tg_expert_ffn_grouped(x_perm, offsets, tiny.S, 80, tiny.w13, tiny.w2, d, I, h, y)
    torch.cuda.synchronize()
    Y = u16(y)
    assert np.array_equal(Y[13 + 13:13 + 40], Y[53:80]), "slot 3 vs its shadow slot 9"
    ref = O.expert_ffn(u16(x_perm[13:53]), u16(tiny.w13[3]), u16(tiny.w2[3]))[1]
    G.assert_close_bf16(Y[13:53], ref, "y slot 3")


def test_ffn_tile_shapes_give_identical_bits(tiny):
    """32-row and 256-row tiles (forced, and the launch's own choice) give
    the same bits on the same rows, across full tiles and ragged tails."""
    d, I, S = tiny.d, tiny.I, tiny.S
    cnt = torch.tensor([0, 33, 1, 70, 0, 64, 31, 40, 29, 32], dtype=torch.int32)
    assert cnt.numel() == S
    P = int(cnt.sum())
    g = torch.Generator().manual_seed(7)
    x_perm = torch.randn((P, d), generator=g).to(torch.bfloat16).to(DEV)
    offsets = torch.zeros(S + 1, dtype=torch.int32)
    offsets[1:] = torch.cumsum(cnt, 0)
    offsets = offsets.to(DEV)
    outs = []
    for policy in (tg.TILES_SMALL, tg.TILES_FULL, tg.TILES_AUTO):
        h = torch.zeros((P, I), dtype=torch.bfloat16, device=DEV)
        y = torch.zeros((P, d), dtype=torch.bfloat16, device=DEV)
        with tg.tile_policy(policy):
            tg.tg_expert_ffn_grouped(x_perm, offsets, S, P, tiny.w13, tiny.w2, d, I, h, y)
        torch.cuda.synchronize()
        outs.append((u16(h), u16(y)))
    for o in outs[1:]:
        assert np.array_equal(outs[0][0], o[0]), "h differs between tile shapes"
        assert np.array_equal(outs[0][1], o[1]), "y differs between tile shapes"
    o = int(offsets[3])
    ref = O.expert_ffn(u16(x_perm[o:o + 70]), u16(tiny.w13[3]), u16(tiny.w2[3]))[1]
    G.assert_close_bf16(outs[0][1][o:o + 70], ref, "y slot 3")


def test_small_tiles_with_partial_last_panels_give_identical_bits():
    """d = 320 and I = 192, multiples of 64 but not of the panel widths: in
    32-row tiles the down projection's last 128-column tile of a slot holds
    64 valid columns and the one after it none, and the gate/up projection's
    last panel is partial too. Forced 32-row tiles, forced 256-row tiles and
    the launch's own choice give the same bits on ragged slots, and every
    row matches the oracle."""
    d, I = 320, 192
    wl = synth.make_custom(T=64, d=d, E=8, k=2, I=I, n_local=8, shadow_experts=[0, 5],
                           gate="weights", seed=23, device=DEV)
    S = wl.S
    cnt = torch.tensor([0, 33, 1, 70, 0, 64, 31, 40, 29, 32], dtype=torch.int32)
    assert cnt.numel() == S
    P = int(cnt.sum())
    g = torch.Generator().manual_seed(9)
    x_perm = torch.randn((P, d), generator=g).to(torch.bfloat16).to(DEV)
    offsets = torch.zeros(S + 1, dtype=torch.int32)
    offsets[1:] = torch.cumsum(cnt, 0)
    off = offsets.numpy()
    offsets = offsets.to(DEV)
    outs = []
    for policy in (tg.TILES_SMALL, tg.TILES_FULL, tg.TILES_AUTO):
        h = torch.zeros((P, I), dtype=torch.bfloat16, device=DEV)
        y = torch.zeros((P, d), dtype=torch.bfloat16, device=DEV)
        with tg.tile_policy(policy):
            tg.tg_expert_ffn_grouped(x_perm, offsets, S, P, wl.w13, wl.w2, d, I, h, y)
        torch.cuda.synchronize()
        outs.append((u16(h), u16(y)))
    for o in outs[1:]:
        assert np.array_equal(outs[0][0], o[0]), "h differs between tile shapes"
        assert np.array_equal(outs[0][1], o[1]), "y differs between tile shapes"
    xp = u16(x_perm)
    for s_ in range(S):
        a, b = int(off[s_]), int(off[s_ + 1])
        if a == b:
            continue
        ref_h, ref_y = O.expert_ffn(xp[a:b], u16(wl.w13[s_]), u16(wl.w2[s_]))
        G.assert_close_bf16(outs[0][0][a:b], ref_h, f"h slot {s_}")
        G.assert_close_bf16(outs[0][1][a:b], ref_y, f"y slot {s_}")


def test_tile_policy_rejects_unknown_values():
    with pytest.raises(tg.TgError):
        tg.tg_set_gemm_tile_policy(3)
    tg.tg_set_gemm_tile_policy(tg.TILES_AUTO)


@pytest.mark.parametrize("big", [700, 1700], ids=["spill16", "spill80"])
def test_ffn_partial_last_round_split_matches_oracle(big):
    """d = 4096 gives the down projection 16 column panels of 256. With 17
    row blocks of 256 (272 tiles) 16 tiles spill past the 256 CUs of one
    round and run as 64 quarter tiles; with 21 row blocks (336 tiles) 80
    spill into 320 quarters, so some blocks take two. Every row is checked
    against the oracle, and the rows of a second layout (the last slot
    empty: 224 tiles without a spill, or 288 tiles with a spill of 32) give
    the same bits."""
    d, I, S = 4096, 128, 10
    counts = [300, 256, 1, 513, 0, 200, 255, 257, big, 530]  # 17 or 21 row blocks of 256
    g = torch.Generator().manual_seed(11)
    x = torch.randn((sum(counts), d), generator=g).to(torch.bfloat16).to(DEV)
    w13 = (torch.randn((S, 2 * I, d), generator=g) * 0.02).to(torch.bfloat16).to(DEV)
    w2 = (torch.randn((S, d, I), generator=g) * 0.02).to(torch.bfloat16).to(DEV)
    ys = []
    for cnt in (counts, counts[:-1] + [0]):
        off = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int32)
        P = int(off[-1])
        h = torch.zeros((P, I), dtype=torch.bfloat16, device=DEV)
        y = torch.zeros((P, d), dtype=torch.bfloat16, device=DEV)
        tg.tg_expert_ffn_grouped(x[:P].contiguous(), torch.from_numpy(off).to(DEV), S, P, w13, w2,
                                 d, I, h, y)
        torch.cuda.synchronize()
        ys.append((off, u16(y)))
    off, Y = ys[0]
    for s in range(S):
        if counts[s]:
            ref = O.expert_ffn(u16(x[off[s]:off[s + 1]]), u16(w13[s]), u16(w2[s]))[1]
            G.assert_close_bf16(Y[off[s]:off[s + 1]], ref, f"y slot {s}")
    n = int(ys[1][0][-1])
    assert np.array_equal(Y[:n], ys[1][1]), "rows differ between layouts with and without a spill"


@pytest.mark.parametrize("tail", [20, 50, 100])
def test_down_spill_in_the_forward_matches_the_standalone_ffn_and_oracle(tail):
    """The down projection's spilled last round, claimed from a counter in
    the fused forward and dealt statically by the standalone FFN entry
    point: 8 slots of 1024 rows and one of 1024 + tail rows give 37 row
    blocks of 16 column panels (d = 4096), two full rounds of 256 tiles and
    a spill of the last slot's 80 tiles. Its full row blocks run as 128-row
    quarters and its tail as 32-, 64- or 128-row pieces (tail = 20, 50,
    100). Routing is exact (one-hot logits, top-1); the two entry points give
    the same bits, and every row matches the oracle."""
    d, I, E = 4096, 128, 9
    counts = [1024] * 8 + [1024 + tail]
    T = sum(counts)
    print(f"[gpu] down spill, tail {tail}: T={T}", flush=True)
    wl = synth.make_custom(T=T, d=d, E=E, k=1, I=I, n_local=E, shadow_experts=[], gate="logits",
                           seed=61 + tail, device=DEV)
    rng = np.random.default_rng(tail)
    assign = rng.permutation(np.repeat(np.arange(E), counts))
    logits = torch.zeros((T, E), dtype=torch.float32)
    logits[torch.arange(T), torch.from_numpy(assign)] = 8.0
    wl.logits = logits.to(DEV)
    f = tg.EwForward(wl, keep_y=True)
    f()
    torch.cuda.synchronize()
    assert np.array_equal(host(f.slot_counts), np.array(counts))
    rows = host(f.pair_row)[:, 0]
    y_fwd = u16(f.y[:T])
    # the same rows in slot order through the standalone entry point
    x_perm = torch.empty_like(wl.x)
    x_perm[torch.from_numpy(rows).long().to(DEV)] = wl.x
    h = torch.empty((T, I), dtype=torch.bfloat16, device=DEV)
    y = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    tg.tg_expert_ffn_grouped(x_perm, f.slot_offsets, wl.S, T, wl.w13, wl.w2, d, I, h, y)
    torch.cuda.synchronize()
    assert np.array_equal(u16(y), y_fwd), "forward (claimed spill) vs standalone (static spill)"
    off = host(f.slot_offsets)
    xp = u16(x_perm)
    for s_ in range(E):
        a, b = int(off[s_]), int(off[s_ + 1])
        ref = O.expert_ffn(xp[a:b], u16(wl.w13[s_]), u16(wl.w2[s_]))[1]
        G.assert_close_bf16(y_fwd[a:b], ref, f"y slot {s_}")


def test_gateup_walk_with_claimed_last_rounds_matches_the_standalone_ffn_and_oracle():
    """With more than six rounds of tiles per XCD, the fused forward deals
    all but the last three statically and claims the rest from counters; the
    standalone FFN entry point deals every tile statically. 8 slots of 610 to
    701 rows (three row blocks each, the last one partial, so the blocks
    drift apart) times 128 gate/up panels (I = 16384, d = 256) give 3072
    tiles, twelve rounds on a 256-CU part. Routing is exact (one-hot logits,
    top-1); the two entry points give the same bits, and every row matches
    the oracle."""
    d, I, E = 256, 16384, 8
    counts = [610 + 13 * i for i in range(E)]
    T = sum(counts)
    print(f"[gpu] gate/up walk with claimed last rounds: T={T}", flush=True)
    wl = synth.make_custom(T=T, d=d, E=E, k=1, I=I, n_local=E, shadow_experts=[], gate="logits",
                           seed=71, device=DEV)
    rng = np.random.default_rng(71)
    assign = rng.permutation(np.repeat(np.arange(E), counts))
    logits = torch.zeros((T, E), dtype=torch.float32)
    logits[torch.arange(T), torch.from_numpy(assign)] = 8.0
    wl.logits = logits.to(DEV)
    f = tg.EwForward(wl, keep_y=True)
    f()
    torch.cuda.synchronize()
    assert np.array_equal(host(f.slot_counts), np.array(counts))
    rows = host(f.pair_row)[:, 0]
    y_fwd = u16(f.y[:T])
    x_perm = torch.empty_like(wl.x)
    x_perm[torch.from_numpy(rows).long().to(DEV)] = wl.x
    h = torch.empty((T, I), dtype=torch.bfloat16, device=DEV)
    y = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    tg.tg_expert_ffn_grouped(x_perm, f.slot_offsets, wl.S, T, wl.w13, wl.w2, d, I, h, y)
    torch.cuda.synchronize()
    assert np.array_equal(u16(y), y_fwd), "forward (claimed last rounds) vs standalone (static)"
    off = host(f.slot_offsets)
    xp = u16(x_perm)
    for s_ in range(E):
        a, b = int(off[s_]), int(off[s_ + 1])
        ref_h, ref_y = O.expert_ffn(xp[a:b], u16(wl.w13[s_]), u16(wl.w2[s_]))
        G.assert_close_bf16(u16(h[a:b]), ref_h, f"h slot {s_}")
        G.assert_close_bf16(y_fwd[a:b], ref_y, f"y slot {s_}")


@pytest.mark.parametrize("extra", [0, 1], ids=["half_round_spilled", "one_more_not_spilled"])
def test_down_spill_threshold_edges_match_oracle(extra):
    """The down projection spills its partial last round when that round
    fills at most half of the grid. With one column panel (d = 256) and full
    row blocks, a last round of exactly half the grid is spilled and one of
    half the grid plus one tile is not; every row matches the oracle on both
    sides of the edge."""
    grid = torch.cuda.get_device_properties(0).multi_processor_count // 8 * 8
    d, I, S = 256, 128, 3
    print(f"[gpu] spill edge, grid {grid}, extra {extra}", flush=True)
    blocks = grid + grid // 2 + extra               # tiles of the down GEMM (one panel)
    split = [blocks // 3, blocks // 3, blocks - 2 * (blocks // 3)]
    counts = [256 * b for b in split]
    g = torch.Generator().manual_seed(71)
    P = sum(counts)
    x = torch.randn((P, d), generator=g).to(torch.bfloat16).to(DEV)
    w13 = (torch.randn((S, 2 * I, d), generator=g) * 0.05).to(torch.bfloat16).to(DEV)
    w2 = (torch.randn((S, d, I), generator=g) * 0.05).to(torch.bfloat16).to(DEV)
    off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    h = torch.empty((P, I), dtype=torch.bfloat16, device=DEV)
    y = torch.empty((P, d), dtype=torch.bfloat16, device=DEV)
    tg.tg_expert_ffn_grouped(x, torch.from_numpy(off).to(DEV), S, P, w13, w2, d, I, h, y)
    torch.cuda.synchronize()
    Y = u16(y)
    for s_ in range(S):
        a, b = int(off[s_]), int(off[s_ + 1])
        ref = O.expert_ffn(u16(x[a:b]), u16(w13[s_]), u16(w2[s_]))[1]
        G.assert_close_bf16(Y[a:b], ref, f"y slot {s_} (grid {grid}, extra {extra})")


def test_persistent_walk_matches_small_tiles_bitwise():
    """Forty slots, every other one empty, with row counts around the tile
    edges (1, 31, 32, 33, 255, 256, 257, ...). With 256-row tiles the
    persistent walk runs 320 gate/up tiles over the CUs (more than one per
    block, across the empty slots) and all of the down GEMM's tiles as tail
    quarters; with 32-row tiles each block walks its range of those. Both,
    and the launch's own choice, give the same bits and the oracle's
    values."""
    d, I, S = 1024, 2560, 40
    base = [0, 1, 31, 32, 33, 255, 256, 257, 0, 0, 2, 63, 64, 65, 100, 0, 17, 5, 1, 0]
    counts = [c for b in base for c in (b, 0)]
    P = sum(counts)
    assert len(counts) == S
    assert sum((c + 255) // 256 for c in counts) * (2 * I // 256) == 320
    g = torch.Generator().manual_seed(21)
    x = torch.randn((P, d), generator=g).to(torch.bfloat16).to(DEV)
    w13 = (torch.randn((S, 2 * I, d), generator=g) * 0.02).to(torch.bfloat16).to(DEV)
    w2 = (torch.randn((S, d, I), generator=g) * 0.02).to(torch.bfloat16).to(DEV)
    off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    offd = torch.from_numpy(off).to(DEV)
    res = []
    for policy in (tg.TILES_SMALL, tg.TILES_FULL, tg.TILES_AUTO):
        h = torch.zeros((P, I), dtype=torch.bfloat16, device=DEV)
        y = torch.zeros((P, d), dtype=torch.bfloat16, device=DEV)
        with tg.tile_policy(policy):
            tg.tg_expert_ffn_grouped(x, offd, S, P, w13, w2, d, I, h, y)
        torch.cuda.synchronize()
        res.append((u16(h), u16(y)))
    for r in res[1:]:
        assert np.array_equal(res[0][0], r[0]), "h: 256-row vs 32-row tiles"
        assert np.array_equal(res[0][1], r[1]), "y: 256-row vs 32-row tiles"
    for s_ in (10, 12, 14, 28):
        a, b = int(off[s_]), int(off[s_ + 1])
        ref = O.expert_ffn(u16(x[a:b]), u16(w13[s_]), u16(w2[s_]))[1]
        G.assert_close_bf16(res[1][1][a:b], ref, f"y slot {s_}")


@pytest.mark.parametrize("name", ["dsv3_decode", "mixtral_small"])
def test_fused_forward_tile_policies_give_identical_bits(name):
    """The fused forward (gathered rows read in place) under each tile
    height: 32-row tiles everywhere, 256-row tiles everywhere and the
    launch's own choice give the same per-pair outputs and outputs, which
    match the oracle on every row."""
    if name == "mixtral_small":
        wl = synth.make_custom(T=96, d=4096, E=8, k=2, I=14336, n_local=8, shadow_experts=[2],
                               gate="weights", seed=5, device=DEV)
    else:
        wl = synth.make(name, device=DEV)
    print(f"[gpu] tile policies on {name}", flush=True)
    res = []
    for policy in (tg.TILES_SMALL, tg.TILES_FULL, tg.TILES_AUTO):
        with tg.tile_policy(policy):
            f = tg.EwForward(wl, keep_y=True)
            f()
            torch.cuda.synchronize()
        P = int(f.slot_offsets[-1])
        res.append((u16(f.y[:P]), u16(f.out), host(f.pair_row)))
        del f
    for r in res[1:]:
        assert np.array_equal(res[0][2], r[2])
        assert np.array_equal(res[0][0], r[0]), "y differs between tile policies"
        assert np.array_equal(res[0][1], r[1]), "out differs between tile policies"
    ref = _oracle_full(wl)
    G.assert_close_bf16(res[2][0], ref["y"], "y (every row)")
    G.assert_out_close(res[2][1], ref, "out (every token)")


def test_repeat_calls_are_bit_identical(tiny):
    a, b = G.run_fused(tiny), G.run_fused(tiny)
    for key in a:
        assert np.array_equal(np.asarray(a[key]), np.asarray(b[key])), key


@pytest.mark.parametrize("T,E,k", [(64, 64, 8), (64, 256, 16), (5000, 64, 8), (5000, 200, 1),
                                   (5000, 256, 8), (4096, 256, 16), (4100, 130, 5)])
def test_logits_topk_ties_and_signed_zeros(T, E, k):
    """Logits mode with many equal logits (including -0 next to +0 and whole
    rows of one value): ids must follow (larger first, equal -> lower id)
    exactly, weights within 1e-6, for small batches (one token per wave) and
    large ones (four tokens per wave)."""
    print(f"[gpu] top-k ties T={T} E={E} k={k}", flush=True)
    rng = np.random.default_rng(T * 7 + E * 3 + k)
    vals = np.array([-2.0, -0.5, -0.0, 0.0, 0.25, 1.0, 3.0], dtype=np.float32)
    logits = vals[rng.integers(0, len(vals), size=(T, E))]
    logits[::17] = 0.25                      # rows of one value
    logits[5::23, : E // 2] = -0.0           # -0 and +0 side by side
    logits[5::23, E // 2:] = 0.0
    lg = torch.from_numpy(logits).to(DEV)
    ids = torch.empty((T, k), dtype=torch.int32, device=DEV)
    w = torch.empty((T, k), dtype=torch.float32, device=DEV)
    tg.tg_gate_topk(None, None, lg, T, 256, E, k, None, ids, w)
    torch.cuda.synchronize()
    ref_ids = O.topk(logits, k)
    assert np.array_equal(host(ids), ref_ids), "top-k ids differ from the oracle"
    ref_w = O.gate_weights(logits, ref_ids)
    assert np.abs(host(w).astype(np.float64) - ref_w).max() <= G.W_ATOL


# ---------------------------------------------------------------- random shapes and edge cases

RANDOM_CASES = [
    # T, d, E, k, I, n_local, shadows, gate, seed
    (1, 256, 8, 2, 128, 8, [0], "weights", 101),
    (37, 512, 16, 4, 384, 12, [1, 5, 11], "weights", 102),
    (200, 256, 64, 6, 256, 20, [0, 7], "logits", 103),
    (513, 256, 8, 1, 128, 8, [], "weights", 104),
    (300, 768, 256, 8, 128, 32, [3, 4, 30], "logits", 105),
    (129, 256, 40, 32, 128, 40, [39], "logits", 106),
    (1000, 256, 4, 4, 128, 4, [2, 2], "weights", 107),   # k = E; two shadows of one expert
    (1024, 256, 16, 4, 128, 12, [3], "weights", 111),    # 4096 pairs: the one-block dispatch's limit
    (77, 192, 16, 3, 320, 16, [4], "weights", 108),      # d, I off the panel grid
    (700, 448, 12, 2, 192, 12, [0, 11], "weights", 109),
    (2731, 256, 24, 3, 128, 20, [2, 9], "logits", 110),  # 8193 pairs: ragged last dispatch chunk
    (150, 2048, 20, 2, 128, 16, [1], "weights", 112),    # gate matrix staged as bf16 (80 KB)
    (150, 1024, 32, 2, 128, 16, [1], "weights", 113),    # gate matrix staged as float32 (128 KB)
]


@pytest.mark.parametrize("case", RANDOM_CASES, ids=[f"T{c[0]}_E{c[2]}_k{c[3]}" for c in RANDOM_CASES])
def test_random_shapes_match_oracle(case):
    T, d, E, k, I, n_local, shadows, gate, seed = case
    print(f"[gpu] random case {case}", flush=True)
    wl = synth.make_custom(T=T, d=d, E=E, k=k, I=I, n_local=n_local, shadow_experts=shadows,
                           gate=gate, seed=seed, device=DEV)
    rng = np.random.default_rng(seed)
    alive = wl.alive.clone()
    dead = rng.choice(wl.S, size=wl.S // 4, replace=False)
    alive[torch.from_numpy(dead).to(DEV)] = 0
    for al in (wl.alive, alive):
        g = G.run_stepwise(wl, al)
        r = _oracle_full(wl, al)
        if g["logits"] is not None:
            assert np.array_equal(g["logits"], r["logits"])
        G.assert_routing_equal(g, r)
        assert np.array_equal(g["x_perm"], r["x_perm"])
        G.assert_close_bf16(g["h"], r["h"], "h")
        G.assert_close_bf16(g["y"], r["y"], "y")
        G.assert_close_bf16(g["out"], r["out"], "out")
        # the fused forward reads token rows in place (gathered); same bits
        f = G.run_fused(wl, al)
        assert np.array_equal(f["out"], g["out"]), "fused differs from stepwise"


@pytest.mark.parametrize("gate,T", [("logits", 200), ("weights", 64)])
def test_largest_supported_shapes_match_oracle(gate, T):
    """The ABI's limits: E = 1024 experts, k = 32, S = 1024 slots (1000
    primaries and 24 shadows: slot indices need 10 bits), routing exact and
    outputs within tolerance, with and without a quarter of the slots
    failed."""
    print(f"[gpu] largest shapes gate={gate} T={T}", flush=True)
    shadows = list(range(0, 1000, 42))[:24]
    wl = synth.make_custom(T=T, d=256, E=1024, k=32, I=128, n_local=1000, shadow_experts=shadows,
                           gate=gate, seed=111, device=DEV)
    assert wl.S == 1024
    rng = np.random.default_rng(112)
    alive = wl.alive.clone()
    alive[torch.from_numpy(rng.choice(wl.S, size=wl.S // 4, replace=False)).to(DEV)] = 0
    for al in (wl.alive, alive):
        g = G.run_stepwise(wl, al)
        r = _oracle_full(wl, al)
        if g["logits"] is not None:
            assert np.array_equal(g["logits"], r["logits"])
        G.assert_routing_equal(g, r)
        G.assert_close_bf16(g["out"], r["out"], "out")
        f = G.run_fused(wl, al)
        assert np.array_equal(f["out"], g["out"]), "fused differs from stepwise"


@pytest.mark.parametrize("d,I,T", [(320, 192, 64), (320, 192, 256), (2880, 2880, 256)],
                         ids=["d320_I192_small", "d320_I192_persistent", "d2880_I2880_persistent"])
def test_widths_off_the_panel_grid_match_oracle(d, I, T):
    """d and I multiples of 64 but not of the weight panels (256 output
    columns for the down projection, 128 gate + 128 up for gate/up): each
    slot's last panel is partial. Routing exact, outputs within tolerance,
    stepwise and fused calls identical, and the shadow failover run
    bit-identical; T=64 takes the 32-row tiles, T=256 the persistent ones."""
    print(f"[gpu] off-grid widths d={d} I={I} T={T}", flush=True)
    wl = synth.make_custom(T=T, d=d, E=8, k=2, I=I, n_local=8, shadow_experts=[0, 5],
                           gate="weights", seed=21, device=DEV, fail_experts=[5])
    g = G.run_stepwise(wl)
    r = _oracle_full(wl)
    assert np.array_equal(g["logits"], r["logits"])
    G.assert_routing_equal(g, r)
    G.assert_close_bf16(g["h"], r["h"], "h")
    G.assert_close_bf16(g["y"], r["y"], "y")
    G.assert_close_bf16(g["out"], r["out"], "out")
    f = G.run_fused(wl)
    assert np.array_equal(f["out"], g["out"]), "fused differs from stepwise"
    fo = G.run_fused(wl, wl.alive_after_failure())
    assert np.array_equal(fo["out"], f["out"]), "failover output differs"


def test_down_spill_with_a_partial_last_panel_matches_oracle():
    """d = 320: the down projection has two column panels per slot, the
    second holding 64 valid columns. 130 row blocks make 260 tiles, so 4
    spill into 16 quarter tiles; the quarters of the second panel's right
    half have no valid column and are skipped. Every row is checked against
    the oracle."""
    d, I, S = 320, 192, 10
    counts = [3300] * 9 + [3280]  # 13 row blocks of 256 each
    g = torch.Generator().manual_seed(23)
    P = sum(counts)
    x = torch.randn((P, d), generator=g).to(torch.bfloat16).to(DEV)
    w13 = (torch.randn((S, 2 * I, d), generator=g) * 0.02).to(torch.bfloat16).to(DEV)
    w2 = (torch.randn((S, d, I), generator=g) * 0.02).to(torch.bfloat16).to(DEV)
    off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    h = torch.zeros((P, I), dtype=torch.bfloat16, device=DEV)
    y = torch.full((P, d), 7, dtype=torch.int16, device=DEV).view(torch.bfloat16)
    tg.tg_expert_ffn_grouped(x, torch.from_numpy(off).to(DEV), S, P, w13, w2, d, I, h, y)
    torch.cuda.synchronize()
    Y = u16(y)
    for s in range(S):
        hr, yr = O.expert_ffn(u16(x[off[s]:off[s + 1]]), u16(w13[s]), u16(w2[s]))
        G.assert_close_bf16(u16(h[off[s]:off[s + 1]]), hr, f"h slot {s}")
        G.assert_close_bf16(Y[off[s]:off[s + 1]], yr, f"y slot {s}")


def _sweep_cases(seed, n):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        E = int(rng.integers(1, 65))
        k = int(rng.integers(1, min(E, 8) + 1))
        n_local = int(rng.integers(1, E + 1))
        T = int(rng.choice([1, 2, 7, 33, 64, 129, 300, 600, 1500]))
        d, I = int(rng.integers(2, 17)) * 64, int(rng.integers(2, 13)) * 64
        shadows = sorted(rng.choice(n_local, size=min(int(rng.integers(0, 4)), n_local)).tolist())
        gate = "weights" if rng.random() < 0.5 else "logits"
        out.append((T, d, E, k, I, n_local, shadows, gate, int(rng.integers(1 << 30)),
                    float(rng.random())))
    return out


@pytest.mark.parametrize("case", _sweep_cases(11, 24), ids=lambda c: f"T{c[0]}_d{c[1]}_E{c[2]}_k{c[3]}_I{c[4]}")
def test_seeded_random_sweep_matches_oracle(case):
    """A seeded sweep over T, d, I (multiples of 64), E, k, local experts,
    shadows and gating mode, each run healthy and with a random set of dead
    slots: routing exact, outputs within tolerance, fused equal to stepwise."""
    T, d, E, k, I, n_local, shadows, gate, seed, p_fail = case
    print(f"[gpu] sweep case {case}", flush=True)
    wl = synth.make_custom(T=T, d=d, E=E, k=k, I=I, n_local=n_local, shadow_experts=shadows,
                           gate=gate, seed=seed, device=DEV)
    rng = np.random.default_rng(seed)
    alive = wl.alive.clone()
    if wl.S > 1 and p_fail < 0.7:
        dead = rng.choice(wl.S, size=int(rng.integers(1, wl.S)), replace=False)
        alive[torch.from_numpy(dead).to(DEV)] = 0
    for al in (wl.alive, alive):
        g = G.run_stepwise(wl, al)
        r = _oracle_full(wl, al)
        if g["logits"] is not None:
            assert np.array_equal(g["logits"], r["logits"])
        G.assert_routing_equal(g, r)
        G.assert_close_bf16(g["out"], r["out"], "out")
        f = G.run_fused(wl, al)
        assert np.array_equal(f["out"], g["out"]), "fused differs from stepwise"


def _ragged_cases(seed, n):
    """Slot populations of four kinds: decode-like (0-39 rows), within three
    rows of a multiple of 256, heavy-tailed (Pareto), and uniform up to 1500;
    T x max(d, I) kept under 2e8 elements."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        E = int(rng.integers(1, 65))
        d = int(rng.choice([128, 256, 320, 512, 768, 1024, 1536, 2048, 4096]))
        I = int(rng.integers(2, 129)) * 64
        while E * 3 * I * d > 6e8:
            I = max(128, I // 128 * 64)
            if I == 128 and E * 3 * I * d > 6e8:
                E = max(1, E // 2)
        kind = int(rng.integers(0, 4))
        if kind == 0:
            counts = rng.integers(0, 40, size=E)
        elif kind == 1:
            counts = 256 * rng.integers(0, 5, size=E) + rng.integers(-3, 4, size=E)
        elif kind == 2:
            counts = (rng.pareto(1.2, size=E) * 300).astype(int)
        else:
            counts = rng.integers(0, 1500, size=E)
        counts = np.clip(counts, 0, 4000).astype(int)
        while counts.sum() * max(I, d) > 2e8:
            counts = counts // 2
        if counts.sum() == 0:
            counts[rng.integers(0, E)] = 1
        out.append((E, d, I, tuple(int(c) for c in counts), int(rng.integers(0, 3)),
                    int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("case", _ragged_cases(5, 12),
                         ids=lambda c: f"E{c[0]}_d{c[1]}_I{c[2]}_T{sum(c[3])}_pol{c[4]}")
def test_ragged_slot_populations_give_identical_bits_under_every_schedule(case):
    """Seeded slot populations of up to 64 slots and 4000 rows each, with the
    routing forced (one-hot logits, top-1). The fused forward (its tile
    policy drawn per case; the last rounds of large launches claimed from
    counters) and the standalone FFN under each of the three tile policies
    (every tile dealt statically) give the same bits; sampled rows of four
    slots, the first and last row of each included, match the oracle."""
    E, d, I, counts, pol, seed = case
    T = sum(counts)
    print(f"[gpu] ragged case E={E} d={d} I={I} T={T} policy={pol}", flush=True)
    wl = synth.make_custom(T=T, d=d, E=E, k=1, I=I, n_local=E, shadow_experts=[], gate="logits",
                           seed=seed, device=DEV)
    rng = np.random.default_rng(seed)
    assign = rng.permutation(np.repeat(np.arange(E), counts))
    logits = torch.zeros((T, E), dtype=torch.float32)
    logits[torch.arange(T), torch.from_numpy(assign)] = 8.0
    wl.logits = logits.to(DEV)
    with tg.tile_policy(pol):
        f = tg.EwForward(wl, keep_y=True)
        f()
        torch.cuda.synchronize()
    assert np.array_equal(host(f.slot_counts), np.array(counts))
    rows = host(f.pair_row)[:, 0]
    y_fwd = u16(f.y[:T])
    x_perm = torch.empty_like(wl.x)
    x_perm[torch.from_numpy(rows).long().to(DEV)] = wl.x
    h = torch.empty((T, I), dtype=torch.bfloat16, device=DEV)
    y = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    for p2 in (tg.TILES_AUTO, tg.TILES_SMALL, tg.TILES_FULL):
        with tg.tile_policy(p2):
            y.zero_()
            tg.tg_expert_ffn_grouped(x_perm, f.slot_offsets, wl.S, T, wl.w13, wl.w2, d, I, h, y)
            torch.cuda.synchronize()
        assert np.array_equal(u16(y), y_fwd), f"forward (policy {pol}) vs standalone (policy {p2})"
    off = host(f.slot_offsets)
    xp, H = u16(x_perm), u16(h)
    for s_ in rng.choice(E, size=min(E, 4), replace=False):
        a, b = int(off[s_]), int(off[s_ + 1])
        if b == a:
            continue
        pick = np.unique(np.concatenate([[a, b - 1], rng.integers(a, b, size=6)]))
        ref_h, ref_y = O.expert_ffn(xp[pick], u16(wl.w13[s_]), u16(wl.w2[s_]))
        G.assert_close_bf16(H[pick], ref_h, f"h slot {s_}")
        G.assert_close_bf16(y_fwd[pick], ref_y, f"y slot {s_}")


def test_empty_batch():
    wl = synth.make_custom(T=4, d=256, E=8, k=2, I=128, n_local=8, shadow_experts=[],
                           gate="weights", seed=5, device=DEV)
    S = wl.S
    buf = torch.full((64,), 5, dtype=torch.int32, device=DEV)
    counts, offsets, nu = buf[:S], buf[16:16 + S + 1], buf[40:41]
    ids = torch.zeros((8, 2), dtype=torch.int32, device=DEV)
    ws = tg.workspace(tg.tg_remap_dispatch_workspace(0, 2, S), DEV)
    tg.tg_remap_dispatch(ids, 0, 2, wl.ert, 8, wl.R, wl.alive, S, wl.x, 256, ids, counts, offsets,
                         ids, ids, wl.x, nu, ws, ws.numel())
    out = wl.x.clone()
    args = tg.make_ew_args(0, 256, 8, 2, 128, S, wl.R, wl.x, wl.wg, None, wl.ert, wl.alive, wl.w13,
                           wl.w2, out)
    wsb = tg.tg_ew_forward_workspace(args)
    tg.tg_ew_forward(args, tg.workspace(wsb, DEV), wsb)
    torch.cuda.synchronize()
    assert host(counts).tolist() == [0] * S and host(offsets).tolist() == [0] * (S + 1)
    assert int(nu[0]) == 0
    assert torch.equal(out, wl.x)  # nothing written for T = 0


def test_all_slots_dead_gives_zero_output_and_counts_every_pair():
    wl = synth.make_custom(T=50, d=256, E=8, k=2, I=128, n_local=8, shadow_experts=[1],
                           gate="weights", seed=6, device=DEV)
    alive = torch.zeros_like(wl.alive)
    f = G.run_fused(wl, alive)
    assert f["n_unserved"] == 100
    assert (f["pair_row"] == -1).all() and f["offsets"][-1] == 0
    assert (f["out"] == 0).all()


def test_share_with_no_local_experts_routes_nothing():
    wl = synth.make_custom(T=64, d=256, E=16, k=2, I=128, n_local=4, shadow_experts=[],
                           gate="logits", seed=7, device=DEV)
    ert = torch.full_like(wl.ert, -1)  # this EW hosts nothing that is selected
    ert[:4, 0] = torch.arange(4, dtype=torch.int32, device=DEV)
    wl.logits[:, :4] = -30.0
    wl.ert = ert
    f = G.run_fused(wl)
    assert f["offsets"][-1] == 0 and f["n_unserved"] == 0 and (f["out"] == 0).all()


# ---------------------------------------------------------------- ERT rows with several candidates

def _junk_ert(wl, width, seed):
    """The workload's ERT widened to ``width`` columns: each expert keeps its
    valid candidates in order, with entries outside [0, S) (-5, -1, S,
    S + 7, 2^30, -2^31) inserted before, between and after them."""
    rng = np.random.default_rng(seed)
    ert = host(wl.ert)
    S = wl.S
    junk = [-5, -1, S, S + 7, 1 << 30, -(1 << 31)]
    out = np.full((wl.E, width), -1, np.int32)
    for e in range(wl.E):
        row = [int(c) for c in ert[e] if 0 <= c < S]
        while len(row) < width:
            row.insert(int(rng.integers(0, len(row) + 1)), junk[int(rng.integers(len(junk)))])
        out[e] = row
    wl.ert = torch.from_numpy(out).to(DEV)
    wl.R = width


def _leading_deaths(wl, experts, n_dead):
    """Liveness with the first n_dead valid candidates of each of ``experts``
    dead (their later candidates stay alive)."""
    ert = host(wl.ert)
    alive = wl.alive.clone()
    for e in experts:
        cands = [int(c) for c in ert[e] if 0 <= c < wl.S]
        for c in cands[:n_dead]:
            alive[c] = 0
    return alive


def _check_masks(wl, masks, bit_identical):
    """Routing exact and outputs within tolerance for every mask; the masks
    in ``bit_identical`` leave every expert a live candidate, so their
    output must equal the all-alive output bit for bit."""
    base = None
    for i, al in enumerate(masks):
        g = G.run_stepwise(wl, al)
        r = _oracle_full(wl, al)
        G.assert_routing_equal(g, r)
        G.assert_close_bf16(g["out"], r["out"], f"out, mask {i}")
        f = G.run_fused(wl, al)
        assert np.array_equal(f["out"], g["out"]), "fused differs from stepwise"
        if i == 0:
            base = f["out"]
        elif i in bit_identical:
            assert np.array_equal(f["out"], base), f"mask {i}: rerouted output differs"
    return base


@pytest.mark.parametrize("T", [500, 3000], ids=["one_block_2000_pairs", "three_grids_12000_pairs"])
def test_ert_with_several_candidates_and_out_of_range_entries(T):
    """Experts with up to five candidates (a primary and up to four shadow
    copies), the ERT padded to eight columns with entries outside [0, S)
    around the valid ones. Leading valid candidates of the shadowed experts
    die (the first two, or the primary only where there is one shadow; then
    the first four of experts 0 and 9): each pair must go to the first live
    candidate past them (§4.2, §5.1) with the output unchanged bit for bit;
    then every candidate of expert 9 dies (its pairs become unserved).
    Covers both dispatch paths (at most 4096 pairs in one block, else three
    grids)."""
    print(f"[gpu] several ERT candidates T={T}", flush=True)
    shadows = [0, 0, 0, 0, 3, 3, 9, 9, 9, 9, 12]
    wl = synth.make_custom(T=T, d=256, E=16, k=4, I=128, n_local=16, shadow_experts=shadows,
                           gate="weights", seed=121, device=DEV)
    assert wl.R == 5  # experts 0 and 9: a primary and four shadows
    _junk_ert(wl, 8, seed=122)
    m2 = _leading_deaths(wl, [0, 3, 9], 2) & _leading_deaths(wl, [12], 1)
    m4 = _leading_deaths(wl, [0, 9], 4)
    m_all = _leading_deaths(wl, [9], 5)
    _check_masks(wl, [wl.alive, m2, m4, m_all], bit_identical={1, 2})
    f = G.run_fused(wl, m_all)
    ids = f["ids"]
    assert f["n_unserved"] == int((ids == 9).sum()) > 0


@pytest.mark.parametrize("T", [100, 300], ids=["one_block_3200_pairs", "three_grids_9600_pairs"])
def test_ert_width_16_at_1024_experts(T):
    """The largest ERT the one-block dispatch stages in LDS: E = 1024 experts
    by R = 16 candidates. Expert 7 has 16 candidates (a primary and 15
    shadows), experts 100 and 500 have 6 and 5; logits are biased so that
    they are chosen often. With the first 15 candidates of expert 7 dead its
    pairs reach its 16th candidate, bit-identically; other rows carry
    entries outside [0, S) in their padding."""
    print(f"[gpu] ERT width 16, E=1024, T={T}", flush=True)
    shadows = [7] * 15 + [100] * 5 + [500] * 4
    wl = synth.make_custom(T=T, d=256, E=1024, k=32, I=128, n_local=1000,
                           shadow_experts=shadows, gate="logits", seed=131, device=DEV)
    assert wl.S == 1024 and wl.R == 16
    wl.logits[:, [7, 100, 500]] += 4.0
    ert = host(wl.ert)
    rng = np.random.default_rng(132)
    pad = ert == -1
    ert[pad] = rng.choice(np.array([-5, 1024, 1031, 1 << 30, -1], np.int32), size=int(pad.sum()))
    wl.ert = torch.from_numpy(ert).to(DEV)
    m15 = _leading_deaths(wl, [7], 15)
    m_mix = _leading_deaths(wl, [7, 100, 500], 4)
    _check_masks(wl, [wl.alive, m15, m_mix], bit_identical={1, 2})
    f = G.run_fused(wl, m15)
    assert f["counts"][7] == 0 and f["counts"][1023 - 9] > 0  # the 16th candidate of expert 7


# ---------------------------------------------------------------- full-size workloads

FULL = ["mixtral", "dsv3_share", "dsv3_skew", "dsv3_decode"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_every_row_matches_oracle(name):
    """The four full-size workloads through the fused forward (the production
    path: gathered rows read in place, persistent tile walks at K = 4096,
    7168, 14336 and 2048): routing exact on every token; every per-pair
    expert output y within tolerance of the oracle; every output element
    within tolerance of the oracle's combine of the kernel's y, and of the
    oracle's own output with the relative part taken against the summed
    terms (see assert_out_close); and the run with failed primaries rerouted
    to shadows bit-identical to the healthy run."""
    print(f"[gpu] full-size {name}", flush=True)
    wl = synth.make(name, device=DEV)
    alive_f = wl.alive_after_failure() if wl.fail_experts else wl.alive_after_failure(
        [wl.slot_expert[wl.S - 1]])  # with no scripted failure, fail the last shadowed expert
    f0 = tg.EwForward(wl, keep_y=True)
    f0()
    f1 = tg.EwForward(wl, alive_f)
    f1()
    torch.cuda.synchronize()
    g0 = dict(ids=host(f0.topk_ids), w=host(f0.topk_w), pair_slot=host(f0.pair_slot),
              counts=host(f0.slot_counts), offsets=host(f0.slot_offsets),
              pair_row=host(f0.pair_row), n_unserved=int(f0.n_unserved[0]), out=u16(f0.out))
    P = int(g0["offsets"][-1])
    y0 = u16(f0.y[:P])
    g1 = dict(ids=host(f1.topk_ids), w=host(f1.topk_w), pair_slot=host(f1.pair_slot),
              counts=host(f1.slot_counts), offsets=host(f1.slot_offsets),
              pair_row=host(f1.pair_row), n_unserved=int(f1.n_unserved[0]), out=u16(f1.out))
    del f0, f1
    assert np.array_equal(g0["out"], g1["out"]), "failure run differs from no-failure run"
    assert g0["counts"].sum() == g1["counts"].sum()
    r1 = O.route(**G.np_inputs(wl, alive_f))
    G.assert_routing_equal(g1, r1, check_perm=False)
    print(f"[gpu] {name}: P={P}, failure run bit-identical; oracle on every row", flush=True)
    r0 = _oracle_full(wl)
    G.assert_routing_equal(g0, r0, check_perm=False)
    G.assert_close_bf16(y0, r0["y"], f"{name} y (all {P} rows)")
    # the combine on the kernel's own y and weights: elementwise
    G.assert_close_bf16(g0["out"], O.combine(y0, g0["pair_row"], g0["w"].astype(np.float64)),
                        f"{name} out vs the oracle's combine of the kernel's y")
    # end to end against the oracle (relative part against the summed terms)
    n_cancel = G.assert_out_close(g0["out"], r0, f"{name} out (all {wl.T} tokens)")
    print(f"[gpu] {name}: every row within tolerance; {n_cancel} of {g0['out'].size} out "
          f"elements outside the plain elementwise bound (cancellation)", flush=True)
