"""The output comparison used against full-size workloads (CPU only).

The end-to-end check of out takes the relative part of the 2e-2 / 1e-2
tolerance against the size of the summed terms, sum_j |w_j y_j|, because the
per-pair outputs y are rounded to bf16 before the combine: a one-ulp
difference in a large y (float32 against float64 accumulation rounding to
neighbouring bf16 values) reaches out whole when the terms cancel. These
tests show that the check accepts exactly that and still rejects the
mistakes it is there to catch.
"""
import numpy as np
import pytest

from oracle import moe_ew as O
from paper_2601_01310_amd import synth
from tests import _gpu as G
from tests._util import u16


@pytest.fixture(scope="module")
def ref():
    wl = synth.make_custom(T=256, d=256, E=8, k=2, I=1024, n_local=8, shadow_experts=[],
                           gate="weights", seed=51, device="cpu")
    # weights scaled by powers of two (exact in bf16): per-pair outputs of
    # the size of the largest ones at the Mixtral shapes (|y| up to 8 and
    # beyond, where one bf16 ulp is 1/16), so that atol hides nothing
    wl.w13.mul_(4)
    wl.w2.mul_(16)
    a = G.np_inputs(wl)
    r = O.ew_forward(**a, w13=u16(wl.w13), w2=u16(wl.w2))
    return r


def _recombine(r, y=None, pair_row=None, w=None):
    return O.combine(r["y"] if y is None else y, r["pair_row"] if pair_row is None else pair_row,
                     r["w"] if w is None else w)


def test_oracle_output_passes_its_own_check(ref):
    assert G.assert_out_close(ref["out"], ref, "self") == 0
    assert np.abs(O.bf16_to_f64(ref["y"])).max() > 8.0


def test_one_ulp_of_a_large_y_under_cancellation_is_accepted(ref):
    """The case met at the Mixtral shapes: one per-pair output of magnitude
    at least 16 rounds to its neighbouring bf16 value (one ulp, 1/8) in a
    token whose terms nearly cancel. The plain elementwise bound rejects
    that out element; the bound against the summed terms accepts it."""
    r = ref
    yf = O.bf16_to_f64(r["y"])
    outf = np.abs(O.bf16_to_f64(r["out"]))
    best = None
    for j in range(r["pair_row"].shape[1]):
        rows = r["pair_row"][:, j]
        big = (np.abs(yf[rows]) >= 16) & (r["w"][:, j] >= 0.3)[:, None] & (outf < 2)
        for t, c in zip(*np.nonzero(big)):
            if best is None or outf[t, c] < outf[best[0], best[1]]:
                best = (t, c, j)
    assert best is not None
    t, c, j = best
    y = r["y"].copy()
    y[r["pair_row"][t, j], c] += 1  # the magnitude's neighbouring bf16 value
    out = _recombine(r, y=y)
    plain_err = abs(O.bf16_to_f64(out[t, c]) - O.bf16_to_f64(r["out"][t, c]))
    assert plain_err > G.ATOL + G.RTOL * outf[t, c]  # the plain bound rejects it
    assert G.assert_out_close(out, r, "one y one ulp off") >= 1


@pytest.mark.parametrize("mistake", ["dropped_term", "swapped_weights", "scale_5pct",
                                     "wrong_rank_row"])
def test_plausible_mistakes_are_rejected(ref, mistake):
    r = ref
    if mistake == "dropped_term":
        pr = r["pair_row"].copy()
        pr[::3, 1] = -1
        out = _recombine(r, pair_row=pr)
    elif mistake == "swapped_weights":
        out = _recombine(r, w=r["w"][:, ::-1].copy())
    elif mistake == "scale_5pct":
        out = O.f64_to_bf16(O.bf16_to_f64(r["out"]) * 1.05)
    else:  # each token's second pair reads its first pair's row
        pr = r["pair_row"].copy()
        pr[:, 1] = pr[:, 0]
        out = _recombine(r, pair_row=pr)
    with pytest.raises(AssertionError):
        G.assert_out_close(out, r, mistake)
