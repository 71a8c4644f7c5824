"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: library
routines for special cases, exact rational arithmetic, brute force on tiny
inputs, closed forms, and the invariants the paper states (stateless,
deterministic experts, §2.1 and §5.1; shadows carry the primary's weights,
§5.3; the MoE output is the gate-weighted sum of the selected experts, §2.1).
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch

from oracle import kv_checkpoint as K
from oracle import moe_ew as O
from paper_2601_01310_amd import synth
from tests._util import bf16_bits_to_f32, host, u16, ulp_diff_bf16

RNG = np.random.default_rng(12345)


def rand_bf16(shape, scale=1.0, rng=RNG):
    return O.f64_to_bf16(rng.standard_normal(shape) * scale)


# ---------------------------------------------------------------- bf16 rounding


def test_bf16_widen_then_round_is_identity():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    f = bf16_bits_to_f32(bits)
    finite = np.isfinite(f)
    back = O.f64_to_bf16(O.bf16_to_f64(bits[finite]))
    assert np.array_equal(back, bits[finite])


def test_bf16_rounding_matches_torch_on_float32_values():
    # torch rounds float32 -> bfloat16 to nearest-even: a library routine that
    # must agree with the oracle on every float32-representable input.
    rng = np.random.default_rng(7)
    v = np.concatenate([
        rng.standard_normal(200000).astype(np.float32),
        (rng.standard_normal(20000) * 1e-39).astype(np.float32),  # subnormals
        # exact bf16 midpoints: a bf16 value plus half its spacing
        (bf16_bits_to_f32(rng.integers(0x0080, 0x7F00, 20000).astype(np.uint16)).view(np.uint32)
         + np.uint32(0x8000)).view(np.float32),
    ])
    ref = u16(torch.from_numpy(v).to(torch.bfloat16))
    got = O.f64_to_bf16(v.astype(np.float64))
    assert np.array_equal(got, ref)


def test_bf16_rounds_once_from_float64():
    # 1 + 2^-8 + 2^-40 lies above the midpoint between 1 and 1 + 2^-7, so it
    # rounds up; a detour through float32 would drop 2^-40 and round to even.
    cases = {
        1.0 + 2.0 ** -8 + 2.0 ** -40: 0x3F81,
        1.0 + 2.0 ** -8: 0x3F80,          # tie -> even
        1.0 + 3 * 2.0 ** -8: 0x3F82,      # tie -> even
        -0.0: 0x8000,
        2.0 ** -133: 0x0001,              # smallest subnormal
        3.0 * 2.0 ** -134: 0x0002,        # subnormal tie -> even
        float("inf"): 0x7F80,
        -1e39: 0xFF80,
    }
    for v, want in cases.items():
        assert int(O.f64_to_bf16(np.array([v]))[0]) == want, v


# ---------------------------------------------------------------- gate logits


def _exact_to_f32(fr: Fraction) -> np.float32:
    """Nearest float32 to a rational, ties to even (by exact comparison)."""
    c = np.float32(float(fr))
    best = None
    for cand in (np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))):
        dist = abs(Fraction(float(cand)) - fr)
        key = (dist, int(np.array(cand).view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, cand)
    return best[1]


def test_gate_logits_are_correctly_rounded_exact_dot_products():
    T, E, d = 6, 5, 97
    x = rand_bf16((T, d))
    wg = rand_bf16((E, d), 0.02)
    got = O.gate_logits(x, wg)
    xf, wf = O.bf16_to_f64(x), O.bf16_to_f64(wg)
    for t in range(T):
        for e in range(E):
            exact = sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(xf[t], wf[e]))
            assert got[t, e] == _exact_to_f32(exact)


def test_gate_logits_one_hot_picks_a_weight_column():
    d, E = 64, 8
    wg = rand_bf16((E, d), 0.02)
    x = np.zeros((d, d), np.uint16)
    x[np.arange(d), np.arange(d)] = 0x3F80  # bf16 1.0
    got = O.gate_logits(x, wg)
    assert np.array_equal(got, bf16_bits_to_f32(wg).T)


# ---------------------------------------------------------------- top-k and weights


@pytest.mark.parametrize("E,k", [(6, 1), (6, 2), (6, 6), (8, 2), (16, 8)])
def test_topk_matches_brute_force_with_ties(E, k):
    rng = np.random.default_rng(E * 10 + k)
    logits = rng.integers(-3, 4, size=(300, E)).astype(np.float32)  # many ties
    got = O.topk(logits, k)
    for t in range(logits.shape[0]):
        want = sorted(range(E), key=lambda e: (-float(logits[t, e]), e))[:k]
        assert list(got[t]) == want


def test_topk_orders_by_float32_not_by_rounding_of_probabilities():
    # two logits one float32 ulp apart must be ordered, even though their
    # probabilities would be equal after float32 rounding of the softmax
    a = np.float32(1.0)
    b = np.nextafter(a, np.float32(2.0))
    got = O.topk(np.array([[a, b, -5.0]], np.float32), 2)
    assert list(got[0]) == [1, 0]


def test_gate_weights_sum_to_one_and_match_topk_softmax():
    rng = np.random.default_rng(3)
    logits = rng.standard_normal((500, 256)).astype(np.float32)
    ids = O.topk(logits, 8)
    w = O.gate_weights(logits, ids)
    assert np.allclose(w.sum(axis=1), 1.0, atol=1e-12, rtol=0)
    # softmax over all E renormalised over the chosen k == softmax over the chosen logits
    chosen = np.take_along_axis(logits.astype(np.float64), ids.astype(np.int64), axis=1)
    assert np.allclose(w, scipy.special.softmax(chosen, axis=1), atol=1e-14, rtol=0)
    assert np.all(np.diff(w, axis=1) <= 0)  # larger logit first -> non-increasing weights


def test_gate_weights_special_cases():
    logits = np.array([[0.5, 2.0, 2.0, -1.0]], np.float32)
    ids = O.topk(logits, 1)
    assert O.gate_weights(logits, ids)[0, 0] == 1.0
    ids2 = O.topk(logits, 2)
    assert list(ids2[0]) == [1, 2]
    assert list(O.gate_weights(logits, ids2)[0]) == [0.5, 0.5]


# ---------------------------------------------------------------- remap


def _tables():
    # E=6 logical experts; this EW holds experts 0..3 as slots 0..3 and shadows
    # of experts 1 and 3 as slots 4, 5; experts 4, 5 live elsewhere.
    ert = np.full((6, 2), -1, np.int32)
    ert[:4, 0] = np.arange(4)
    ert[1, 1] = 4
    ert[3, 1] = 5
    return ert


def test_remap_all_alive_uses_primaries_and_skips_remote_experts():
    ert = _tables()
    rng = np.random.default_rng(0)
    ids = np.stack([rng.permutation(6)[:3] for _ in range(50)]).astype(np.int32)
    ps, nu = O.remap(ids, ert, np.ones(6, np.uint8))
    want = np.where(ids < 4, ids, -1)
    assert np.array_equal(ps, want) and nu == 0


def test_remap_dead_primary_moves_exactly_its_pairs_to_the_shadow():
    ert = _tables()
    rng = np.random.default_rng(1)
    ids = np.stack([rng.permutation(6)[:3] for _ in range(80)]).astype(np.int32)
    alive = np.ones(6, np.uint8)
    base, _ = O.remap(ids, ert, alive)
    alive[3] = 0
    ps, nu = O.remap(ids, ert, alive)
    assert nu == 0
    assert np.array_equal(ps[ids == 3], np.full((ids == 3).sum(), 5))
    assert np.array_equal(ps[ids != 3], base[ids != 3])


def test_remap_no_live_candidate_counts_unserved():
    ert = _tables()
    ids = np.array([[0, 1, 4], [2, 0, 5], [1, 3, 0]], np.int32)
    alive = np.ones(6, np.uint8)
    alive[[0, 1, 4]] = 0  # expert 0 has no replica; expert 1 loses both
    ps, nu = O.remap(ids, ert, alive)
    assert nu == 5  # experts 0 and 1 have local candidates, none alive: 2 + 1 + 2 pairs
    assert ps.tolist() == [[-1, -1, -1], [2, -1, -1], [-1, 3, -1]]


def test_remap_ignores_out_of_range_table_entries():
    ert = np.array([[7, 1], [-5, -1]], np.int32)  # slot 7 does not exist (S=2)
    ps, nu = O.remap(np.array([[0, 1]], np.int32), ert, np.ones(2, np.uint8))
    assert ps.tolist() == [[1, -1]] and nu == 0


# ---------------------------------------------------------------- dispatch


def test_dispatch_matches_stable_sort_construction():
    rng = np.random.default_rng(4)
    T, k, S = 300, 4, 7
    ps = rng.integers(-1, S, size=(T, k)).astype(np.int32)
    counts, offsets, perm, pair_row = O.dispatch(ps, S)
    flat = ps.ravel()
    assert np.array_equal(counts, np.bincount(flat[flat >= 0], minlength=S))
    assert offsets[0] == 0 and np.array_equal(np.diff(offsets), counts)
    keyed = np.flatnonzero(flat >= 0)
    want = keyed[np.argsort(flat[keyed], kind="stable")]  # (slot, token, rank) order
    assert np.array_equal(perm, want)
    inv = np.full(T * k, -1)
    inv[perm] = np.arange(len(perm))
    assert np.array_equal(pair_row.ravel(), inv)


def test_dispatch_empty():
    counts, offsets, perm, pair_row = O.dispatch(np.full((5, 2), -1, np.int32), 3)
    assert counts.tolist() == [0, 0, 0] and offsets.tolist() == [0, 0, 0, 0]
    assert perm.size == 0 and (pair_row == -1).all()


# ---------------------------------------------------------------- expert FFN closed forms


def test_swiglu_closed_form_with_identity_and_permutation_weights():
    # W1 = I, W3 = 2I, W2 = a permutation: h = bf16(silu(x) * 2x) and y[c] = h[pi(c)].
    # Swapping the gate and up halves, or transposing W2, changes the result.
    n = 32
    rng = np.random.default_rng(5)
    one, two = 0x3F80, 0x4000
    w13 = np.zeros((2 * n, n), np.uint16)
    w13[np.arange(n), np.arange(n)] = one
    w13[n + np.arange(n), np.arange(n)] = two
    pi = rng.permutation(n)
    w2 = np.zeros((n, n), np.uint16)
    w2[np.arange(n), pi] = one
    x = rand_bf16((40, n), 2.0, rng)
    h, y = O.expert_ffn(x, w13, w2)
    xf = O.bf16_to_f64(x)
    want_h = O.f64_to_bf16(xf * scipy.special.expit(xf) * 2.0 * xf)
    assert np.array_equal(h, want_h)
    assert np.array_equal(y, h[:, pi])


def test_ffn_rows_are_independent_and_w2_scaling_is_exact():
    rng = np.random.default_rng(6)
    d, I = 64, 96
    x = rand_bf16((9, d), 1.0, rng)
    w13 = rand_bf16((2 * I, d), 0.05, rng)
    w2 = rand_bf16((d, I), 0.05, rng)
    h, y = O.expert_ffn(x, w13, w2)
    for r in range(x.shape[0]):  # a row's result does not depend on its batch
        hr, yr = O.expert_ffn(x[r:r + 1], w13, w2)
        assert np.array_equal(hr[0], h[r]) and np.array_equal(yr[0], y[r])
    w2x2 = O.f64_to_bf16(O.bf16_to_f64(w2) * 2.0)
    _, y2 = O.expert_ffn(x, w13, w2x2)
    assert np.array_equal(O.bf16_to_f64(y2), 2.0 * O.bf16_to_f64(y))


def test_ffn_float64_agrees_with_float32_torch_within_bf16_rounding():
    rng = np.random.default_rng(8)
    d, I = 128, 256
    x = rand_bf16((16, d), 1.0, rng)
    w13 = rand_bf16((2 * I, d), 0.02 * 4, rng)
    w2 = rand_bf16((d, I), 0.02 * 4, rng)
    _, y = O.expert_ffn(x, w13, w2)
    xt = torch.from_numpy(bf16_bits_to_f32(x))
    wt = torch.from_numpy(bf16_bits_to_f32(w13))
    g, uu = xt @ wt[:I].T, xt @ wt[I:].T
    ht = (torch.nn.functional.silu(g) * uu).to(torch.bfloat16).float()
    yt = (ht @ torch.from_numpy(bf16_bits_to_f32(w2)).T).to(torch.bfloat16)
    assert ulp_diff_bf16(u16(yt), y).max() <= 2


# ---------------------------------------------------------------- whole forward


def _np_workload(wl):
    return dict(x=host(wl.x), wg=None if wl.wg is None else host(wl.wg),
                logits=None if wl.logits is None else host(wl.logits), k=wl.k,
                ert=host(wl.ert), alive=host(wl.alive), w13=host(wl.w13), w2=host(wl.w2))


@pytest.fixture(scope="module")
def tiny():
    return synth.make("tiny")


def test_dense_mixture_brute_force_tiny(tiny):
    """out[t] = sum over ALL experts e of g~_e * FFN_e(x_t), g~ = renormalised
    gate weight on the top-k and 0 elsewhere (§2.1), evaluated densely with
    torch float64 on every (token, expert) pair and no routing tables."""
    a = _np_workload(tiny)
    r = O.ew_forward(**a)
    x = torch.from_numpy(bf16_bits_to_f32(a["x"]).astype(np.float64))
    wg = torch.from_numpy(bf16_bits_to_f32(a["wg"]).astype(np.float64))
    logits = (x @ wg.T).float()
    T, E, k, I = tiny.T, tiny.E, tiny.k, tiny.I
    p = torch.softmax(logits.double(), dim=1)
    out = torch.zeros(T, tiny.d, dtype=torch.float64)
    for t in range(T):
        chosen = sorted(range(E), key=lambda e: (-float(logits[t, e]), e))[:k]
        z = sum(float(p[t, e]) for e in chosen)
        for e in range(E):  # dense: every expert, gate weight 0 off the top-k
            gw = float(p[t, e]) / z if e in chosen else 0.0
            w13 = torch.from_numpy(bf16_bits_to_f32(a["w13"][e]).astype(np.float64))
            w2 = torch.from_numpy(bf16_bits_to_f32(a["w2"][e]).astype(np.float64))
            g, u = w13[:I] @ x[t], w13[I:] @ x[t]
            h = torch.from_numpy(bf16_bits_to_f32(O.f64_to_bf16(
                (torch.nn.functional.silu(g) * u).numpy())).astype(np.float64))
            y = torch.from_numpy(bf16_bits_to_f32(O.f64_to_bf16((w2 @ h).numpy())).astype(np.float64))
            out[t] += gw * y
    want = O.f64_to_bf16(out.numpy())
    assert ulp_diff_bf16(r["out"], want).max() <= 1
    assert (ulp_diff_bf16(r["out"], want) == 0).mean() > 0.99


def test_failure_run_equals_no_failure_run_bitwise(tiny):
    """Rerouting expert 3 to its shadow (same weights, §5.3) leaves every
    output bit unchanged (replay through a healthy replica is identical, §5.1)."""
    a = _np_workload(tiny)
    r0 = O.ew_forward(**a)
    a["alive"] = host(tiny.alive_after_failure())
    r1 = O.ew_forward(**a)
    assert np.array_equal(r0["out"], r1["out"])
    assert np.array_equal(r0["ids"], r1["ids"])
    moved = r0["ids"] == 3
    assert (r1["pair_slot"][moved] == 9).all() and (r0["pair_slot"][moved] == 3).all()
    assert r1["counts"][3] == 0 and r1["counts"][9] == r0["counts"][3]
    assert r0["counts"].sum() == r1["counts"].sum() == tiny.T * tiny.k


def test_token_permutation_permutes_outputs(tiny):
    a = _np_workload(tiny)
    r0 = O.ew_forward(**a)
    pi = np.random.default_rng(9).permutation(tiny.T)
    a["x"] = a["x"][pi]
    r1 = O.ew_forward(**a)
    assert np.array_equal(r1["out"], r0["out"][pi])
    assert np.array_equal(r1["ids"], r0["ids"][pi])


def test_unserved_pairs_are_dropped_without_renormalising(tiny):
    a = _np_workload(tiny)
    r0 = O.ew_forward(**a)
    a["alive"] = a["alive"].copy()
    a["alive"][[1, 9]] = 0  # expert 1 has no shadow; kill slot 9 too (expert 3's shadow)
    r1 = O.ew_forward(**a)
    assert r1["n_unserved"] == int((r0["ids"] == 1).sum())
    t = np.flatnonzero((r0["ids"] == 1).any(axis=1))[0]
    j_keep = [j for j in range(tiny.k) if r0["ids"][t, j] != 1]
    y0 = O.bf16_to_f64(r0["y"][r0["pair_row"][t, j_keep]])
    want = O.f64_to_bf16((r0["w"][t, j_keep][:, None] * y0).sum(axis=0))
    assert np.array_equal(r1["out"][t], want)


# ---------------------------------------------------------------- partial batch (§5.2)


def test_partial_batch_equals_forward_on_the_included_tokens(tiny):
    """Tokens outside the batch are not routed (pair_slot -2) and get +0; the
    other tokens get exactly what a forward over them alone gives."""
    a = _np_workload(tiny)
    valid = np.random.default_rng(3).random(tiny.T) < 0.6
    a["alive"] = a["alive"].copy()
    a["alive"][1] = 0  # expert 1 unserved: only included tokens may count
    r = O.ew_forward(**a, token_valid=valid)
    rs = O.ew_forward(**dict(a, x=a["x"][valid]))
    assert np.array_equal(r["out"][valid], rs["out"])
    assert not r["out"][~valid].any()
    assert (r["pair_slot"][~valid] == -2).all() and (r["pair_row"][~valid] == -1).all()
    assert np.array_equal(r["pair_slot"][valid], rs["pair_slot"])
    assert r["n_unserved"] == rs["n_unserved"] == int((rs["ids"] == 1).sum()) > 0
    assert np.array_equal(r["counts"], rs["counts"])


def test_batch_trigger_brute_force_over_delivery_and_liveness():
    """Every combination of delivered / healthy flags over 4 AWs (one with an
    empty chunk, one partly past T): the batch is exactly the rows of healthy
    AWs that delivered, and the condition follows the rule of §5.2."""
    chunk_rows = [0, 10, 25, 25, 60]
    T = 48
    rows_of = [10, 15, 0, 23]
    for bits in itertools.product([0, 1], repeat=8):
        delivered, alive = bits[:4], bits[4:]
        for min_rows in (0, 20, 49):
            cond, tv, rows, n = O.batch_trigger(delivered, alive, chunk_rows, T, min_rows)
            inc = [a for a in range(4) if delivered[a] and alive[a]]
            want = np.zeros(T, dtype=np.uint8)
            for a in inc:
                want[chunk_rows[a]:min(chunk_rows[a + 1], T)] = 1
            assert np.array_equal(tv, want) and rows == int(want.sum()) == sum(rows_of[a] for a in inc)
            assert n == len(inc)
            everyone = all(delivered[a] for a in range(4) if alive[a])
            assert cond == (0 if everyone else 1 if rows >= min_rows else 2)


def test_batch_trigger_agrees_with_the_arrival_process():
    """§5.2 as a process in time: AWs deliver their chunks one after another
    (seeded random order, some never), failure detection can mark AWs
    unhealthy at any moment, and the EW starts at the first moment when
    every AW still healthy has delivered, or else when the rows buffered
    from healthy AWs reach the minimum, or else when the probe window ends.
    At each event before that moment the snapshot rule must say "not yet"
    (condition 2 with the window still open); at the starting moment it must
    give the reason the process started for (all delivered has priority over
    the minimum when both happen at the same event), and the batch must hold
    exactly the rows delivered so far by healthy AWs."""
    rng = np.random.default_rng(77)
    for trial in range(400):
        A = int(rng.integers(1, 7))
        sizes = rng.integers(0, 30, A)
        chunk_rows = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
        T = int(chunk_rows[-1] + rng.integers(-10, 5))
        T = max(T, 0)
        rows_in = [min(max(int(chunk_rows[a + 1]), 0), T) - min(max(int(chunk_rows[a]), 0), T)
                   for a in range(A)]
        min_rows = int(rng.integers(0, max(2, sum(rows_in) + 5)))
        # events: ("d", a) a delivery, ("f", a) a failure detection; some AWs never deliver
        events = [("d", a) for a in range(A) if rng.random() < 0.8]
        events += [("f", a) for a in range(A) if rng.random() < 0.25]
        rng.shuffle(events)
        window = int(rng.integers(0, len(events) + 2))  # the probe window ends after this many events
        delivered = np.zeros(A, np.uint8)
        alive = np.ones(A, np.uint8)
        started = None
        for i in range(len(events) + 1):
            if i > 0:
                kind, a = events[i - 1]
                if kind == "d":
                    delivered[a] = 1
                else:
                    alive[a] = 0
            healthy = [a for a in range(A) if alive[a]]
            everyone = all(delivered[a] for a in healthy)
            have = sum(rows_in[a] for a in healthy if delivered[a])
            reason = 0 if everyone else 1 if have >= min_rows else None
            if reason is None and i >= window:
                reason = 2
            cond, tv, rows, n = O.batch_trigger(delivered, alive, chunk_rows, T, min_rows)
            if reason is None:
                assert cond == 2, (trial, i)
                continue
            started = (reason, cond, tv, rows, n, delivered.copy(), alive.copy())
            break
        if started is None:  # every event seen, window still open: the EW waits on
            continue
        reason, cond, tv, rows, n, dl, al = started
        assert cond == reason, (trial, reason, cond)
        want = np.zeros(T, np.uint8)
        for a in range(A):
            if dl[a] and al[a]:
                lo, hi = min(max(int(chunk_rows[a]), 0), T), min(max(int(chunk_rows[a + 1]), 0), T)
                want[lo:hi] = 1
        assert np.array_equal(tv, want) and rows == int(want.sum())
        assert n == int(sum(1 for a in range(A) if dl[a] and al[a]))


# ---------------------------------------------------------------- replay (§5.1)


def _replay(tiny, a, r0, alive, y=None, out=None):
    return O.replay(a["x"], tiny.k, a["ert"], alive, a["w13"], a["w2"], r0["ids"], r0["w"],
                    r0["pair_slot"], r0["pair_row"], r0["y"] if y is None else y,
                    r0["out"] if out is None else out)


def _lost_outputs(r, slot):
    """Outputs of ``slot`` that never arrived: its y rows and the out rows of
    its tokens hold NaN."""
    y, out = r["y"].copy(), r["out"].copy()
    hit = r["pair_slot"] == slot
    y[r["pair_row"][hit]] = 0x7FC0
    out[np.flatnonzero(hit.any(axis=1))] = 0x7FC0
    return y, out


def test_replay_after_a_mid_layer_failure_equals_the_failover_forward(tiny):
    """Slot 3 fails after the first pass: its pairs are recomputed on the
    shadow (slot 9) and the result equals a forward that routed them there
    from the start."""
    a = _np_workload(tiny)
    r0 = O.ew_forward(**a)
    alive1 = host(tiny.alive_after_failure())
    r1 = O.ew_forward(**dict(a, alive=alive1))
    y, out = _lost_outputs(r0, 3)
    out2, rs, n_rep, n_un = _replay(tiny, a, r0, alive1, y, out)
    assert np.array_equal(out2, r1["out"])
    assert np.array_equal(rs >= 0, r0["pair_slot"] == 3) and (rs[rs >= 0] == 9).all()
    assert n_rep == int((r0["pair_slot"] == 3).sum()) > 0
    assert n_un == r1["n_unserved"] == 0


def test_replay_with_nothing_failed_changes_nothing(tiny):
    a = _np_workload(tiny)
    r0 = O.ew_forward(**a)
    out2, rs, n_rep, n_un = _replay(tiny, a, r0, a["alive"])
    assert np.array_equal(out2, r0["out"]) and (rs == -1).all() and n_rep == 0 and n_un == 0


def test_replay_drops_pairs_whose_expert_has_no_live_candidate(tiny):
    """Slot 1 (expert 1, no shadow) fails: its pairs leave the sums, the
    other weights are not renormalised, as in a forward without slot 1."""
    a = _np_workload(tiny)
    r0 = O.ew_forward(**a)
    alive1 = a["alive"].copy()
    alive1[1] = 0
    r1 = O.ew_forward(**dict(a, alive=alive1))
    out2, rs, n_rep, n_un = _replay(tiny, a, r0, alive1)
    assert np.array_equal(out2, r1["out"])
    assert n_rep == 0 and (rs == -1).all()
    assert n_un == r1["n_unserved"] == int((r0["ids"] == 1).sum()) > 0
    untouched = ~(r0["pair_slot"] == 1).any(axis=1)
    assert np.array_equal(out2[untouched], r0["out"][untouched])


def test_replay_computes_pairs_that_had_no_live_candidate(tiny):
    """Expert 3 was unserved (slots 3 and 9 dead); once slot 3 is back its
    pairs are computed and merged."""
    a = _np_workload(tiny)
    alive0 = a["alive"].copy()
    alive0[[3, 9]] = 0
    r0 = O.ew_forward(**dict(a, alive=alive0))
    r1 = O.ew_forward(**a)
    out2, rs, n_rep, n_un = _replay(tiny, a, r0, a["alive"])
    assert np.array_equal(out2, r1["out"])
    assert np.array_equal(rs >= 0, r0["ids"] == 3) and (rs[rs >= 0] == 3).all()
    assert n_rep == r0["n_unserved"] > 0 and n_un == 0


def test_replay_leaves_tokens_outside_the_batch_alone(tiny):
    a = _np_workload(tiny)
    valid = np.random.default_rng(5).random(tiny.T) < 0.5
    r0 = O.ew_forward(**a, token_valid=valid)
    alive1 = host(tiny.alive_after_failure())
    r1 = O.ew_forward(**dict(a, alive=alive1), token_valid=valid)
    y, out = _lost_outputs(r0, 3)
    out2, rs, n_rep, _ = _replay(tiny, a, r0, alive1, y, out)
    assert np.array_equal(out2, r1["out"]) and not out2[~valid].any()
    assert (rs[~valid] == -1).all() and n_rep == int((r0["pair_slot"] == 3).sum())


def test_partial_combines_over_expert_shares_add_up():
    """Each EW of an expert-parallel group sums only its local pairs with the
    global weights; summing the partials of all shares gives the full MoE
    output (within the bf16 rounding of each partial)."""
    E, n_share = 16, 4
    wl = synth.make_custom(T=24, d=64, E=E, k=4, I=96, n_local=E, shadow_experts=[],
                           gate="weights", seed=11)
    a = _np_workload(wl)
    full = O.ew_forward(**a)
    acc = np.zeros((wl.T, wl.d))
    for sh in range(n_share):
        local = list(range(sh * 4, sh * 4 + 4))
        ert = np.full((E, 2), -1, np.int32)
        ert[local, 0] = np.arange(4)
        b = dict(a, ert=ert, alive=np.ones(4, np.uint8), w13=a["w13"][local], w2=a["w2"][local])
        part = O.ew_forward(**b)
        assert part["n_unserved"] == 0
        acc += O.bf16_to_f64(part["out"])
    full_f = O.bf16_to_f64(full["out"])
    assert np.all(np.abs(acc - full_f) <= 4 * 2.0 ** -8 * np.maximum(np.abs(full_f), 1e-3) + 1e-6)


def test_sampled_token_path_equals_full_forward(tiny):
    a = _np_workload(tiny)
    r = O.ew_forward(**a)
    toks = [0, 5, 17, 63]
    ids, w, ps, out = O.ew_forward_tokens(toks, a["x"], a["wg"], a["logits"], a["k"], a["ert"],
                                          a["alive"], lambda s: a["w13"][s], lambda s: a["w2"][s])
    assert np.array_equal(ids, r["ids"][toks]) and np.array_equal(ps, r["pair_slot"][toks])
    assert np.array_equal(out, r["out"][toks])


def test_skewed_workload_sends_about_forty_percent_to_the_four_hottest():
    wl = synth.make("dsv3_skew", with_weights=False)
    ids = O.topk(host(wl.logits), wl.k)
    local = ids[ids < 32]
    share = np.isin(local, wl.hot_experts).mean()
    assert 0.38 <= share <= 0.42, share


# ---------------------------------------------------------------- KV checkpoint (§6.1, §6.2)


def _kv_case(seed=0, size=1 << 16):
    rng = np.random.default_rng(seed)
    kv = rng.integers(0, 256, size=size, dtype=np.uint8)
    return rng, kv


def test_segment_sizes_of_app_c_for_mixtral():
    """Mixtral-8x7B: 8 KV heads of 128 of a 4096 hidden size over 32 heads,
    bf16: a KV segment is 4 KiB, 12.5 % of the 32 KiB of expert traffic."""
    C = K.segment_bytes(8, 4096, 32, 2)
    V = K.expert_traffic_bytes(2, 4096, 2)
    assert C == 4096 and V == 32768 and C / V == 0.125


def test_checkpoint_then_restore_round_trips_committed_segments():
    rng, kv = _kv_case()
    store = np.full(kv.size, 0xEE, dtype=np.uint8)
    log = np.zeros((8, 3), dtype=np.uint64)
    offs = np.array([0, 4096, 512, 60000], dtype=np.uint64)
    nbs = np.array([256, 1024, 16, 5536], dtype=np.uint32)
    store, log, commit = K.checkpoint(kv, store, log, 8, 0, offs, nbs, first_seq=100)
    assert commit == 104
    for o, n in zip(offs.tolist(), nbs.tolist()):
        assert np.array_equal(store[o:o + n], kv[o:o + n])
    touched = np.zeros(kv.size, bool)
    for o, n in zip(offs.tolist(), nbs.tolist()):
        touched[o:o + n] = True
    assert (store[~touched] == 0xEE).all()
    assert log[100 % 8].tolist() == [100, 0, 256] and log[103 % 8].tolist() == [103, 60000, 5536]
    dst = np.zeros(1 << 15, dtype=np.uint8)
    dsts = np.array([0, 256, 1280, 1296], dtype=np.uint64)
    out, st = K.restore(store, commit, np.arange(100, 104), offs, dsts, nbs, dst)
    assert st.tolist() == [1, 1, 1, 1]
    for o, d, n in zip(offs.tolist(), dsts.tolist(), nbs.tolist()):
        assert np.array_equal(out[d:d + n], kv[o:o + n])


def test_uncommitted_segments_are_not_restored():
    """A batch whose commit record never landed (the worker died first) is
    skipped by restoration even though its bytes are in the store."""
    rng, kv = _kv_case(1)
    store = np.zeros(kv.size, dtype=np.uint8)
    log = np.zeros((4, 3), dtype=np.uint64)
    store, log, c1 = K.checkpoint(kv, store, log, 4, 0, [0], [64], first_seq=0)
    kv2 = kv.copy()
    kv2[64:128] ^= 0xFF
    store, log, c2 = K.checkpoint(kv2, store, log, 4, c1, [64], [64], first_seq=1,
                                  write_commit=False)
    assert c2 == c1 == 1
    out, st = K.restore(store, c2, [0, 1], [0, 64], [0, 64], [64, 64], np.zeros(256, np.uint8))
    assert st.tolist() == [1, 0] and np.array_equal(out[:64], kv[:64]) and not out[64:].any()


def test_misaligned_or_out_of_range_segments_are_rejected():
    _, kv = _kv_case(2, size=1024)
    store, log, commit = K.checkpoint(kv, np.zeros(1024, np.uint8), np.zeros((4, 3), np.uint64),
                                      4, 0, [8, 1008, 0], [16, 32, 48], first_seq=0)
    assert log[:3, 2].tolist() == [0, 0, 48] and not store[48:].any()
    _, st = K.restore(store, commit, [2, 2], [0, 0], [0, 1000], [48, 48], np.zeros(1024, np.uint8))
    assert st.tolist() == [1, 2]
