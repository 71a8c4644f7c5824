"""Gate logits on the GPU at float32 rounding midpoints (§2.1, reading R3).

Token and gate rows are built so that each exact dot product lies 2^-40
above, exactly on, or 2^-40 below a float32 midpoint, behind a +1024 /
-1024 pair that a float32 running sum would lose the small terms to; the
expected logits are the correctly rounded values from exact rational
arithmetic. The three weight-mode paths of the gate (matrix staged in LDS
widened to float32, staged as bf16, read from memory) must return them bit
for bit; so must the full-size Mixtral workload as generated on the GPU,
whose every logit rounds the same in any float64 summation order.
"""
import numpy as np
import pytest
import torch

from oracle import moe_ew as O
from paper_2601_01310_amd import synth, tg
from tests import _gate_cases as C
from tests._util import host, u16

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _gate(x_bits, w_bits, k):
    T, d = x_bits.shape
    E = w_bits.shape[0]
    x = torch.from_numpy(x_bits.view(np.int16)).view(torch.bfloat16).to(DEV)
    w = torch.from_numpy(w_bits.view(np.int16)).view(torch.bfloat16).to(DEV)
    logits = torch.empty((T, E), dtype=torch.float32, device=DEV)
    ids = torch.empty((T, k), dtype=torch.int32, device=DEV)
    tw = torch.empty((T, k), dtype=torch.float32, device=DEV)
    tg.tg_gate_topk(x, w, None, T, d, E, k, logits, ids, tw)
    torch.cuda.synchronize()
    return host(logits), host(ids), host(tw)


@pytest.mark.parametrize("T,E,d", [(45, 8, 256), (40, 8, 5120), (37, 16, 4096)],
                         ids=["staged_f32", "staged_bf16", "unstaged"])
def test_logits_at_float32_midpoints_are_correctly_rounded(T, E, d):
    print(f"[gpu] gate midpoints T={T} E={E} d={d}", flush=True)
    x, w, expected, delta = C.engineered(T, E, d, seed=T * 1000 + d)
    k = 2
    logits, ids, tw = _gate(x, w, k)
    bad = logits.view(np.uint32) != expected.view(np.uint32)
    assert not bad.any(), (f"{int(bad.sum())} of {bad.size} logits not correctly rounded "
                           f"(offsets {sorted(set(delta[bad].tolist()))})")
    r_ids = O.topk(expected, k)
    assert np.array_equal(ids, r_ids)
    assert np.abs(tw - O.gate_weights(expected, r_ids)).max() <= 1e-6


def test_full_size_mixtral_logits_are_correctly_rounded_by_construction():
    """The Mixtral workload (4096 tokens, d = 4096, 8 experts) as generated
    on the GPU: every logit rounds the same in any float64 summation order
    (checked exactly on the host), and the kernel's logits equal the
    oracle's bit for bit."""
    print("[gpu] gate: full-size mixtral exactness", flush=True)
    wl = synth.make("mixtral", device=DEV, with_weights=False)
    xb, wb = u16(wl.x), u16(wl.wg)
    ok, exact, worst = C.rounding_is_order_independent(xb, wb)
    assert ok.all(), f"{int((~ok).sum())} logits could round either way"
    print(f"[gpu] mixtral: {int(exact.sum())} of {exact.size} exact float64 sums; "
          f"the rest >= {worst:.3g} x the float64 error bound from a midpoint", flush=True)
    logits, _, _ = _gate(xb, wb, wl.k)
    assert np.array_equal(logits.view(np.uint32), O.gate_logits(xb, wb).view(np.uint32))
