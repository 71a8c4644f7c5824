"""CPU oracle for the Tarragon expert-worker (EW) forward (arXiv 2601.01310).

TEST INFRASTRUCTURE ONLY. This module is the slow, plain definition that the
HIP path is checked against. Only the tests, the smoke check and the CPU
baseline leg of the benchmark may import it; the product path never does. It
shares no code with the HIP path: it reads numpy arrays (bf16 as uint16) and
computes with numpy in float64.

What is computed, per token t of one MoE layer (§2.1; §4.2; §5.1; §5.3):

1. gate logits  l[t, e] = sum_i x[t, i] * Wg[e, i], returned as the float32
   nearest to the float64 dot product (bf16 x bf16 products are exact in
   float64, so this is the correctly rounded logit up to a 2^-53 relative
   error), or logits given directly;
2. top-k       the k largest float32 logits, larger first, ties to the lower
   expert id;
3. weights     softmax over all E logits, renormalised over the chosen k (the
   gating weights of the weighted sum, §2.1), in float64;
4. remap       each chosen logical expert resolves through the ERT to the
   first candidate slot that is alive (§4.2 decouples identity from
   location; a failed primary is replaced by a healthy replica or a shadow,
   §5.1, §5.3); -1 if the expert has no live local candidate;
5. dispatch    per-slot counts, exclusive offsets, and the permutation of the
   routed pairs in (slot, token, rank) order (the EW batches tokens per
   expert, §2.2.1);
6. expert FFN  SwiGLU: h = bf16(silu(x W1^T) * (x W3^T)), y = bf16(h W2^T),
   sums in float64 (experts are stateless pure functions of their input,
   §2.1);
7. combine     out[t] = bf16(sum over the token's routed pairs, in rank order,
   of w * y), +0 when the token has no routed pair here (gate-weighted sum,
   §2.1).

Beyond the single forward (§5.1, §5.2):

8. partial batch  tokens outside the batch (their attention worker has not
   delivered, §5.2) are not routed and get +0; ``batch_trigger`` decides
   which workers' tokens form the batch;
9. replay         after a forward, pairs whose slot has failed are rerouted
   to the next live candidate, recomputed from the same token row and merged
   into the output (§5.1).

Readings where the paper is silent (each listed in the design notes): the
SwiGLU form and layouts, the bf16 rounding points of h, y and out, the
tie-break, the permutation order, first-alive replica choice, partial combine
over one share with the global weights, and the fp32 logit precision.

Every function here has a pin in ``tests/test_oracle.py``.
"""

from __future__ import annotations

import numpy as np

# ----------------------------------------------------------------------------
# bf16 <-> float64 (bf16 is the top half of an IEEE binary32)
# ----------------------------------------------------------------------------


def bf16_to_f64(u16: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to float64 exactly."""
    u16 = np.asarray(u16, dtype=np.uint16)
    return (u16.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float64 to the nearest bf16, ties to even, in one rounding step.

    A finite value is written m * 2^e with m in [0.5, 1); bf16 keeps 8
    significant bits, so the result is rint(m * 256) * 2^(e - 8), except
    below 2^-126 where bf16 spacing is fixed at 2^-133. Values beyond the
    largest bf16 after rounding become +-inf; NaN stays NaN.
    """
    a = np.asarray(a, dtype=np.float64)
    out = np.empty(a.shape, dtype=np.float64)
    finite = np.isfinite(a)
    m, e = np.frexp(a[finite])
    q = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)
    small = np.abs(a[finite]) < 2.0 ** -126
    q[small] = np.rint(a[finite][small] * 2.0 ** 133) * 2.0 ** -133
    big = np.abs(q) > 3.3895313892515355e38  # largest finite bf16
    q[big] = np.copysign(np.inf, q[big])
    out[finite] = q
    out[~finite] = a[~finite]
    bits = out.astype(np.float32).view(np.uint32)  # exact: q has <= 8 significant bits
    res = (bits >> 16).astype(np.uint16)
    res[np.isnan(out)] = 0x7FC0
    return res


# ----------------------------------------------------------------------------
# 1-3. gating (§2.1)
# ----------------------------------------------------------------------------


def gate_logits(x: np.ndarray, wg: np.ndarray) -> np.ndarray:
    """Gate logits l[t, e] = x[t] . Wg[e], float64 sum, rounded once to float32."""
    return (bf16_to_f64(x) @ bf16_to_f64(wg).T).astype(np.float32)


def topk(logits: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest logits per row, larger first; equal logits -> lower id."""
    logits = np.asarray(logits, dtype=np.float32)
    T, E = logits.shape
    ids = np.empty((T, k), dtype=np.int32)
    eid = np.arange(E)
    for t in range(T):
        order = np.lexsort((eid, -logits[t].astype(np.float64)))  # primary key last
        ids[t] = order[:k]
    return ids


def gate_weights(logits: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Softmax over all E logits, then renormalised over the chosen k (float64)."""
    l64 = np.asarray(logits, dtype=np.float32).astype(np.float64)
    p = np.exp(l64 - l64.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    chosen = np.take_along_axis(p, ids.astype(np.int64), axis=1)
    return chosen / chosen.sum(axis=1, keepdims=True)


# ----------------------------------------------------------------------------
# 4. ERT remap with failure mask (§4.2, §5.1, §5.3)
# ----------------------------------------------------------------------------


def remap(ids: np.ndarray, ert: np.ndarray, alive: np.ndarray, token_valid=None):
    """pair_slot[t, j] = first candidate c of ert[ids[t, j]] with 0 <= c < S and alive[c].

    A pair whose expert lists at least one valid local candidate, none alive,
    is counted in ``n_unserved`` (it must be replayed on another EW); an
    expert with no valid local candidate belongs to another EW and is not
    counted. Entries outside [0, S) are ignored. Tokens with
    ``token_valid[t] == 0`` are not in this batch (the EW started without
    them, §5.2): their pairs get -2 and are not counted.
    """
    T, k = ids.shape
    S = alive.shape[0]
    pair_slot = np.full((T, k), -1, dtype=np.int32)
    n_unserved = 0
    for t in range(T):
        if token_valid is not None and not token_valid[t]:
            pair_slot[t] = -2
            continue
        for j in range(k):
            cands = [int(c) for c in ert[ids[t, j]] if 0 <= int(c) < S]
            live = [c for c in cands if alive[c]]
            if live:
                pair_slot[t, j] = live[0]
            elif cands:
                n_unserved += 1
    return pair_slot, n_unserved


# ----------------------------------------------------------------------------
# 5. per-slot batching: counts, offsets, permutation (§2.2.1, §5.2)
# ----------------------------------------------------------------------------


def dispatch(pair_slot: np.ndarray, S: int):
    """Counts, exclusive offsets [S+1], perm (flat pair ids t*k+j in (slot, token,
    rank) order) and pair_row[t, j] (row of the pair in the permuted batch, -1
    if not routed here)."""
    T, k = pair_slot.shape
    rows = [[] for _ in range(S)]
    for t in range(T):
        for j in range(k):
            s = pair_slot[t, j]
            if s >= 0:
                rows[s].append(t * k + j)
    counts = np.array([len(r) for r in rows], dtype=np.int32)
    offsets = np.zeros(S + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    perm = np.array([p for r in rows for p in r], dtype=np.int32)
    pair_row = np.full((T, k), -1, dtype=np.int32)
    for r, p in enumerate(perm):
        pair_row[p // k, p % k] = r
    return counts, offsets, perm, pair_row


# ----------------------------------------------------------------------------
# 6. expert FFN (SwiGLU) and 7. combine (§2.1)
# ----------------------------------------------------------------------------


def silu(g: np.ndarray) -> np.ndarray:
    return g / (1.0 + np.exp(-g))


def _ffn_f64(xf: np.ndarray, w13f: np.ndarray, w2f: np.ndarray):
    I = w13f.shape[0] // 2
    g = xf @ w13f[:I].T
    u = xf @ w13f[I:].T
    h = f64_to_bf16(silu(g) * u)
    y = f64_to_bf16(bf16_to_f64(h) @ w2f.T)
    return h, y


def expert_ffn(x_rows: np.ndarray, w13: np.ndarray, w2: np.ndarray):
    """SwiGLU expert on bf16 rows: returns (h, y) as bf16 bit patterns.

    x_rows [M, d], w13 [2I, d] (gate rows then up rows), w2 [d, I]; each row
    of the result depends only on its own input row.
    """
    return _ffn_f64(bf16_to_f64(x_rows), bf16_to_f64(w13), bf16_to_f64(w2))


def combine(y: np.ndarray, pair_row: np.ndarray, w: np.ndarray) -> np.ndarray:
    """out[t] = bf16(sum_j w[t, j] * y[pair_row[t, j]]) over routed pairs, rank order."""
    T, k = pair_row.shape
    d = y.shape[1] if y.ndim == 2 else 0
    yf = bf16_to_f64(y)
    out = np.zeros((T, d), dtype=np.float64)
    for t in range(T):
        for j in range(k):
            r = pair_row[t, j]
            if r >= 0:
                out[t] = out[t] + w[t, j] * yf[r]
    return f64_to_bf16(out)


# ----------------------------------------------------------------------------
# the whole EW forward
# ----------------------------------------------------------------------------


def route(x, wg, logits, k, ert, alive, token_valid=None):
    """Steps 1-5: returns a dict with logits, ids, w, pair_slot, n_unserved,
    counts, offsets, perm, pair_row."""
    if logits is None:
        logits = gate_logits(x, wg)
    logits = np.asarray(logits, dtype=np.float32)
    ids = topk(logits, k)
    w = gate_weights(logits, ids)
    pair_slot, n_unserved = remap(ids, ert, alive, token_valid)
    counts, offsets, perm, pair_row = dispatch(pair_slot, alive.shape[0])
    return dict(logits=logits, ids=ids, w=w, pair_slot=pair_slot, n_unserved=n_unserved,
                counts=counts, offsets=offsets, perm=perm, pair_row=pair_row)


def ew_forward(x, wg, logits, k, ert, alive, w13, w2, token_valid=None):
    """The full EW forward on all tokens (or on the tokens marked in
    ``token_valid``). Returns the routing dict plus x_perm, h, y (bf16, in
    permuted row order) and out [T, d] (bf16)."""
    r = route(x, wg, logits, k, ert, alive, token_valid)
    T, d = x.shape
    I = w13.shape[1] // 2
    P = int(r["offsets"][-1])
    x_perm = x[r["perm"] // k] if P else np.zeros((0, d), np.uint16)
    h = np.zeros((P, I), dtype=np.uint16)
    y = np.zeros((P, d), dtype=np.uint16)
    for s in range(alive.shape[0]):
        a, b = int(r["offsets"][s]), int(r["offsets"][s + 1])
        if b > a:
            h[a:b], y[a:b] = expert_ffn(x_perm[a:b], w13[s], w2[s])
    r.update(x_perm=x_perm, h=h, y=y, out=combine(y, r["pair_row"], r["w"]))
    return r


def ew_forward_tokens(tokens, x, wg, logits, k, ert, alive, w13_of, w2_of):
    """out rows for a subset of tokens, one token at a time (for sampled checks
    at sizes where the full oracle would take too long).

    ``w13_of(s)`` / ``w2_of(s)`` return slot s's weights as uint16 arrays, so
    callers can fetch slots lazily. Returns (ids, w, pair_slot, out) for the
    chosen tokens.
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    xs = x[tokens]
    lg = gate_logits(xs, wg) if logits is None else np.asarray(logits, np.float32)[tokens]
    ids = topk(lg, k)
    w = gate_weights(lg, ids)
    pair_slot, _ = remap(ids, ert, alive)
    n = len(tokens)
    d = x.shape[1]
    y = np.zeros((n, k, d), dtype=np.uint16)
    for s in sorted({int(v) for v in pair_slot.ravel() if v >= 0}):
        w13f, w2f = bf16_to_f64(w13_of(s)), bf16_to_f64(w2_of(s))
        for i in range(n):
            for j in range(k):
                if pair_slot[i, j] == s:
                    y[i, j] = _ffn_f64(bf16_to_f64(xs[i:i + 1]), w13f, w2f)[1][0]
    acc = np.zeros((n, d), dtype=np.float64)
    for i in range(n):
        for j in range(k):
            if pair_slot[i, j] >= 0:
                acc[i] = acc[i] + w[i, j] * bf16_to_f64(y[i, j])
    return ids, w, pair_slot, f64_to_bf16(acc)


# ----------------------------------------------------------------------------
# replay of failed pairs (§5.1)
# ----------------------------------------------------------------------------


def replay(x, k, ert, alive, w13, w2, ids, w, pair_slot, pair_row, y, out):
    """Replays the pairs of a finished forward whose slots have since failed.

    Following §5.1: a pair whose slot is no longer alive is rerouted to the
    next live candidate of its expert (§4.2, §5.3) and recomputed there from
    the same token row; experts are stateless and deterministic (§2.1), so
    the recomputed output is the one the failed slot would have produced. A
    pair that had no live candidate may now have one and is computed too. A
    pair that loses its slot with no live candidate left is dropped (R8: the
    other weights are not renormalised). Every token with a replayed or
    dropped pair gets its output re-formed from its pairs' outputs in rank
    order; other tokens keep their output.

    ``ids``, ``w``, ``pair_slot``, ``pair_row``, ``y`` and ``out`` are the
    first pass's (``ew_forward``'s) results; ``alive`` is the current mask.
    Returns (out, replay_slot [T, k], n_replayed, n_unserved).
    """
    T = ids.shape[0]
    S = alive.shape[0]
    valid = pair_slot[:, 0] != -2 if T else np.zeros(0, bool)
    now_slot, n_unserved = remap(ids, ert, alive, valid)
    replay_slot = np.full((T, k), -1, dtype=np.int32)
    changed = set()
    for t in range(T):
        for j in range(k):
            prior = int(pair_slot[t, j])
            if prior == -2 or (prior >= 0 and alive[prior]):
                continue  # outside the batch, or the first-pass output stands
            if now_slot[t, j] >= 0:
                replay_slot[t, j] = now_slot[t, j]
                changed.add(t)
            elif prior >= 0:
                changed.add(t)  # its slot failed and nothing can take it
    _, offsets, perm, replay_row = dispatch(replay_slot, S)
    n_replayed = int(offsets[-1])
    d = x.shape[1]
    y2 = np.zeros((n_replayed, d), dtype=np.uint16)
    for s in range(S):
        a, b = int(offsets[s]), int(offsets[s + 1])
        if b > a:
            y2[a:b] = expert_ffn(x[perm[a:b] // k], w13[s], w2[s])[1]
    out = np.array(out, dtype=np.uint16, copy=True)
    for t in sorted(changed):
        acc = np.zeros(d, dtype=np.float64)
        for j in range(k):
            if replay_row[t, j] >= 0:
                acc = acc + w[t, j] * bf16_to_f64(y2[replay_row[t, j]])
            elif pair_slot[t, j] >= 0 and alive[pair_slot[t, j]]:
                acc = acc + w[t, j] * bf16_to_f64(y[pair_row[t, j]])
        out[t] = f64_to_bf16(acc)
    return out, replay_slot, n_replayed, n_unserved


# ----------------------------------------------------------------------------
# EW-side partial batch (§5.2)
# ----------------------------------------------------------------------------


def batch_trigger(delivered, aw_alive, chunk_rows, T, min_rows):
    """Which attention workers' tokens form the batch, for a fixed set of
    delivered chunks (§5.2).

    The EW starts when (0) every AW still deemed healthy has delivered, or
    (1) the tokens buffered from healthy AWs reach the minimum batch size;
    otherwise (2) the probing window runs out and the healthy AWs that have
    not delivered are left out of this batch. AW a's tokens are rows
    chunk_rows[a] .. chunk_rows[a+1]-1 of the batch buffer (clipped to
    [0, T)). Returns (condition, token_valid [T] uint8, rows, n_aws).
    """
    A = len(aw_alive)
    got = [bool(aw_alive[a]) and bool(delivered[a]) for a in range(A)]
    spans = []
    for a in range(A):
        lo = min(max(int(chunk_rows[a]), 0), T)
        hi = min(max(int(chunk_rows[a + 1]), lo), T)
        spans.append((lo, hi))
    rows = sum(hi - lo for (lo, hi), g in zip(spans, got) if g)
    if all(got[a] for a in range(A) if aw_alive[a]):
        cond = 0
    elif rows >= min_rows:
        cond = 1
    else:
        cond = 2
    token_valid = np.zeros(T, dtype=np.uint8)
    for (lo, hi), g in zip(spans, got):
        if g:
            token_valid[lo:hi] = 1
    return cond, token_valid, rows, sum(got)
