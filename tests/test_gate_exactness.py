"""The gate logit as the correctly rounded dot product (§2.1, reading R3),
pinned with exact rational arithmetic (CPU only).

A bf16 x bf16 product has at most 16 significant bits; when the sum of
|products| of a logit stays below 2^(53 + e), e the lowest set bit over its
products, every float64 partial sum in any order is exact, so any float64
accumulation rounded once to float32 gives the correctly rounded logit.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import moe_ew as O
from paper_2601_01310_amd import synth
from tests import _gate_cases as C
from tests._util import u16


@pytest.fixture(scope="module")
def cases():
    return C.engineered()


def test_rounding_helper_matches_float64_to_float32_casts():
    """The exact-rational rounding used as the reference agrees with the
    IEEE cast (round to nearest, ties to even) on doubles, ties included."""
    rng = np.random.default_rng(3)
    v = rng.standard_normal(4000) * 2.0 ** rng.integers(-20, 20, 4000)
    f = v.astype(np.float32).astype(np.float64)
    ulp = np.spacing(np.abs(v).astype(np.float32)).astype(np.float64)
    ties = f + np.sign(v) * ulp / 2  # exact midpoints (float64 holds them)
    for a in np.concatenate([v, ties]):
        assert np.float32(float(C.round_f32(Fraction(float(a))))) == np.float32(a)


def test_oracle_logits_are_correctly_rounded_at_midpoints(cases):
    """Exact dot products 2^-40 above, exactly on, and 2^-40 below float32
    midpoints, behind a +1024 / -1024 pair: the oracle's logits are the
    correctly rounded values, bit for bit, and a float32 running sum misses
    every one of them."""
    x, w, expected, delta = cases
    got = O.gate_logits(x, w)
    assert np.array_equal(got.view(np.uint32), expected.view(np.uint32))
    assert {-1, 0, 1} == set(np.unique(delta))
    xf = (x.astype(np.uint32) << 16).view(np.float32)
    wf = (w.astype(np.uint32) << 16).view(np.float32)
    acc = np.zeros(expected.shape, np.float32)
    for i in range(x.shape[1]):
        acc = (acc + np.outer(xf[:, i], wf[:, i])).astype(np.float32)
    assert (acc != expected).all()


def test_midpoint_cases_round_by_their_offset(cases):
    """Above a midpoint rounds away from zero, below rounds towards it, on
    it rounds to the even neighbour."""
    x, w, expected, delta = cases
    xf = [[C.bf16_value(b) for b in row] for row in x]
    wf = [[C.bf16_value(b) for b in row] for row in w]
    for t in range(0, x.shape[0], 7):
        for e in range(w.shape[0]):
            s = sum(a * b for a, b in zip(xf[t], wf[e]))
            r = Fraction(float(expected[t, e]))
            lo = C.round_f32(s - Fraction(1, 2 ** 40) * delta[t, e])  # the midpoint itself
            assert abs(s - r) <= abs(s - Fraction(float(np.nextafter(expected[t, e], 0))))
            if delta[t, e] > 0:
                assert abs(r) > abs(s)
            elif delta[t, e] < 0:
                assert abs(r) < abs(s)
            else:
                bits = int(np.array([expected[t, e]], np.float32).view(np.uint32)[0])
                assert bits % 2 == 0 and r == lo


def test_exactness_margin_flags_order_dependent_sums():
    """A logit whose float64 sum depends on the order (2^60, -2^60 and 1)
    has a non-positive margin; the engineered and ordinary rows do not."""
    x = np.array([[C.bf16_from_dyadic(1, 60), C.bf16_from_dyadic(1, 60), C.W_ONE, 0]], np.uint16)
    w = np.array([[C.W_ONE, C.bf16_from_dyadic(-1, 0), C.W_ONE, 0]], np.uint16)
    assert C.exactness_margin(x, w)[0, 0] <= 0
    p = [2.0 ** 60, -(2.0 ** 60), 1.0]
    assert (p[0] + p[2]) + p[1] != (p[0] + p[1]) + p[2]  # the sum really depends on the order


@pytest.mark.parametrize("name", ["tiny", "mixtral"])
def test_every_logit_of_the_seeded_workloads_rounds_the_same_in_any_order(name):
    """For the weight-gated workloads (x ~ N(0,1), gate rows ~ N(0, 0.02) in
    bf16) every logit is the correctly rounded dot product whatever the
    float64 summation order: nearly all have an exact float64 sum, and the
    few whose products span too many binades lie far from every float32
    midpoint compared with the float64 error bound. Kernel and oracle agree
    on every logit by construction, not by chance."""
    wl = synth.make(name, device="cpu", with_weights=False)
    ok, exact, worst = C.rounding_is_order_independent(u16(wl.x), u16(wl.wg))
    assert ok.all(), f"{int((~ok).sum())} logits could round either way"
    print(f"{name}: {int(exact.sum())} of {exact.size} logits with an exact float64 sum; "
          f"the rest at >= {worst:.3g} x the error bound from a midpoint")
