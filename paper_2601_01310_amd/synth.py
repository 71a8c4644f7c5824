"""Seeded synthetic inputs for the expert-worker (EW) forward.

This module only draws random numbers and lays out tables; it holds none of
the method's arithmetic (no gating, routing, FFN or combine). Both the HIP
path and the CPU oracle take their inputs from here, so the two see the same
bytes.

Workloads (shapes of the paper's evaluation models; weights are random, since
no trained checkpoint is used):

* ``tiny``        T=64, d=256, E=8, top-2, I=512; 8 primary slots plus shadow
                  copies of experts 0 and 3; expert 3's primary fails.
* ``mixtral``     Mixtral-8x7B layer shapes (§7.1 workload): T=4096, d=4096,
                  E=8, top-2, I=14336; shadows of experts 0 and 5; expert 5's
                  primary fails.
* ``dsv3_share``  one expert-parallel share of a DeepSeek-V3 layer (8 of 256
                  experts active per token, §2.1 footnote): T=16384, d=7168,
                  I=2048; this GPU holds logical experts 0..31 as slots 0..31
                  plus 8 shadow slots of seeded local experts; gate logits
                  are given, i.i.d. N(0,1) fp32.
* ``dsv3_skew``   as ``dsv3_share`` with a Zipf(s=1.2) per-expert logit bias
                  over the local experts; shadows cover the 4 hottest local
                  experts plus 4 seeded others; the 4 hottest primaries fail.
* ``dsv3_decode`` as ``dsv3_share`` with T=128 (decode-size batch).

Value recipe: activations bf16 from N(0,1), gate and expert weights bf16 from
N(0, 0.02^2), each drawn as fp32 and rounded to nearest-even bf16. Shadow
slots hold byte copies of their primary's weights (a shadow carries the same
weights as its primary, §5.3).

Expert weights are stored per slot: ``w13[s]`` is ``[2I, d]`` (rows 0..I-1
the gate projection W1, rows I..2I-1 the up projection W3) and ``w2[s]`` is
``[d, I]``; both are (out, in) row-major bf16. The ERT is ``[E, R]`` int32,
candidate slots in priority order (primary first, then the expert's shadows
in slot order), -1 padded; an expert with no local candidate is served by
another EW.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import torch

# Scale of the Zipf logit bias of the skewed workload. Chosen so that the four
# hottest local experts receive close to 40% of the local routed pairs; the
# value was found by ``tests/golden/skew_beta.py`` and is checked by a test.
ZIPF_S = 1.2
ZIPF_BETA = 0.333

CONFIGS: Dict[str, dict] = {
    "tiny": dict(T=64, d=256, E=8, k=2, I=512, n_local=8, gate="weights",
                 shadows=[0, 3], fail=[3], seed=0),
    "mixtral": dict(T=4096, d=4096, E=8, k=2, I=14336, n_local=8, gate="weights",
                    shadows=[0, 5], fail=[5], seed=1),
    "dsv3_share": dict(T=16384, d=7168, E=256, k=8, I=2048, n_local=32, gate="logits",
                       shadows="seeded8", fail=[], seed=2),
    "dsv3_skew": dict(T=16384, d=7168, E=256, k=8, I=2048, n_local=32, gate="logits",
                      shadows="hot4+seeded4", fail="hot4", seed=3, zipf=True),
    "dsv3_decode": dict(T=128, d=7168, E=256, k=8, I=2048, n_local=32, gate="logits",
                        shadows="seeded8", fail=[], seed=4),
}


@dataclasses.dataclass
class Workload:
    name: str
    T: int
    d: int
    E: int
    k: int
    I: int
    S: int
    R: int
    x: torch.Tensor                 # [T, d] bf16
    wg: Optional[torch.Tensor]      # [E, d] bf16, or None when logits are given
    logits: Optional[torch.Tensor]  # [T, E] fp32, or None when gate weights are given
    ert: torch.Tensor               # [E, R] int32
    alive: torch.Tensor             # [S] uint8, all slots alive
    w13: torch.Tensor               # [S, 2I, d] bf16
    w2: torch.Tensor                # [S, d, I] bf16
    slot_expert: List[int]          # logical expert held by each slot
    fail_experts: List[int]         # experts whose primary slot fails in the failure run
    hot_experts: List[int]          # the hottest local experts (skewed workload), else []

    def alive_after_failure(self, experts: Optional[List[int]] = None) -> torch.Tensor:
        """Slot liveness with the primaries of ``experts`` marked dead."""
        experts = self.fail_experts if experts is None else experts
        a = self.alive.clone()
        for e in experts:
            a[int(self.ert[e, 0])] = 0
        return a

    @property
    def device(self) -> torch.device:
        return self.x.device


def _gen(seed: int, stream: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1_000_003 + stream)
    return g


def _bf16_normal(shape, std: float, seed: int, stream: int, device) -> torch.Tensor:
    g = _gen(seed, stream, device)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(torch.bfloat16)


def zipf_bias(E: int, n_local: int, beta: float, seed: int) -> (torch.Tensor, List[int]):
    """Per-expert logit bias over the local experts: beta * (-s*ln r_e - mean).

    r_e is a seeded permutation of 1..n_local over the local experts; experts
    outside this share get bias 0. Returns the bias (fp32 [E], CPU) and the
    local experts ordered hottest first.
    """
    g = _gen(seed, 99, "cpu")
    ranks = torch.randperm(n_local, generator=g) + 1  # rank of local expert e
    raw = torch.tensor([-ZIPF_S * math.log(float(r)) for r in ranks.tolist()], dtype=torch.float64)
    raw -= raw.mean()
    bias = torch.zeros(E, dtype=torch.float64)
    bias[:n_local] = beta * raw
    hottest = sorted(range(n_local), key=lambda e: int(ranks[e]))
    return bias.to(torch.float32), hottest


def make_tables(E: int, n_local: int, shadow_experts: List[int]):
    """ERT [E, R] and slot->expert list: slot e holds local expert e (e < n_local),
    slots n_local.. hold shadow copies of ``shadow_experts`` in order.

    An expert's row lists its primary, then its shadows in slot order, then
    -1; R is 1 + the largest number of shadows of any one expert (§4.2 lets
    an expert map to one or more candidate locations)."""
    S = n_local + len(shadow_experts)
    n_shadow = [0] * E
    for e in shadow_experts:
        n_shadow[e] += 1
    R = 1 + max(n_shadow + [0])
    ert = torch.full((E, R), -1, dtype=torch.int32)
    for e in range(n_local):
        ert[e, 0] = e
    slot_expert = list(range(n_local))
    col = [1] * E
    for i, e in enumerate(shadow_experts):
        ert[e, col[e]] = n_local + i
        col[e] += 1
        slot_expert.append(e)
    return ert, slot_expert, S


def make_custom(T: int, d: int, E: int, k: int, I: int, n_local: int,
                shadow_experts: List[int], gate: str, seed: int, device="cpu",
                fail_experts: Optional[List[int]] = None, logit_bias: Optional[torch.Tensor] = None,
                name: str = "custom", hot_experts: Optional[List[int]] = None,
                with_weights: bool = True) -> Workload:
    """A workload of any shape with the value recipe of the module docstring.

    ``with_weights=False`` leaves ``w13``/``w2`` as empty [S, 0, 0] tensors
    (routing-only studies)."""
    device = torch.device(device)
    ert, slot_expert, S = make_tables(E, n_local, shadow_experts)
    x = _bf16_normal((T, d), 1.0, seed, 1, device)
    wg = logits = None
    if gate == "weights":
        wg = _bf16_normal((E, d), 0.02, seed, 2, device)
    elif gate == "logits":
        g = _gen(seed, 3, device)
        logits = torch.randn((T, E), generator=g, device=device, dtype=torch.float32)
        if logit_bias is not None:
            logits += logit_bias.to(device)[None, :]
    else:
        raise ValueError(gate)
    if not with_weights:
        w13 = torch.empty((S, 0, 0), dtype=torch.bfloat16, device=device)
        w2 = torch.empty((S, 0, 0), dtype=torch.bfloat16, device=device)
        n_local_w = 0
    else:
        w13 = torch.empty((S, 2 * I, d), dtype=torch.bfloat16, device=device)
        w2 = torch.empty((S, d, I), dtype=torch.bfloat16, device=device)
        n_local_w = n_local
    for s in range(n_local_w):
        w13[s] = _bf16_normal((2 * I, d), 0.02, seed, 1000 + 2 * s, device)
        w2[s] = _bf16_normal((d, I), 0.02, seed, 1001 + 2 * s, device)
    for s in range(n_local, S if with_weights else n_local):
        w13[s].copy_(w13[slot_expert[s]])
        w2[s].copy_(w2[slot_expert[s]])
    alive = torch.ones(S, dtype=torch.uint8, device=device)
    return Workload(name=name, T=T, d=d, E=E, k=k, I=I, S=S, R=int(ert.shape[1]), x=x, wg=wg, logits=logits,
                    ert=ert.to(device), alive=alive, w13=w13, w2=w2, slot_expert=slot_expert,
                    fail_experts=list(fail_experts or []), hot_experts=list(hot_experts or []))


def make(name: str, device="cpu", T: Optional[int] = None, with_weights: bool = True) -> Workload:
    """Build a named workload. ``T`` may shrink the token count (same recipe)."""
    c = CONFIGS[name]
    seed = c["seed"]
    n_local = c["n_local"]
    bias = None
    hot: List[int] = []
    if c.get("zipf"):
        bias, order = zipf_bias(c["E"], n_local, ZIPF_BETA, seed)
        hot = order[:4]
    shadows = c["shadows"]
    if isinstance(shadows, str):
        g = _gen(seed, 98, "cpu")
        if shadows == "seeded8":
            shadows = sorted(torch.randperm(n_local, generator=g)[:8].tolist())
        elif shadows == "hot4+seeded4":
            rest = [e for e in torch.randperm(n_local, generator=g).tolist() if e not in hot]
            shadows = list(hot) + sorted(rest[:4])
        else:
            raise ValueError(shadows)
    fail = c["fail"]
    if fail == "hot4":
        fail = list(hot)
    return make_custom(T=T or c["T"], d=c["d"], E=c["E"], k=c["k"], I=c["I"], n_local=n_local,
                       shadow_experts=list(shadows), gate=c["gate"], seed=seed, device=device,
                       fail_experts=fail, logit_bias=bias, name=name, hot_experts=hot,
                       with_weights=with_weights)
