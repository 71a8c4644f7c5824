"""Finds the scale of the Zipf logit bias of the skewed workload.

The skewed workload adds beta * (-1.2 ln r_e - mean) to the N(0,1) logits of
the local experts (r_e a seeded rank 1..32). This script bisects beta until
the four hottest local experts receive 40% of the local routed pairs, using
the oracle's top-k only, and writes the result to ``skew_beta.json``. The
generator's ``ZIPF_BETA`` is that value rounded to three decimals.

Run: python tests/golden/skew_beta.py
"""
import json
import os
import sys

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import moe_ew as O  # noqa: E402
from paper_2601_01310_amd import synth  # noqa: E402


def share(beta: float) -> float:
    c = synth.CONFIGS["dsv3_skew"]
    bias, order = synth.zipf_bias(c["E"], c["n_local"], beta, c["seed"])
    wl = synth.make_custom(T=c["T"], d=8, E=c["E"], k=c["k"], I=8, n_local=c["n_local"],
                           shadow_experts=[], gate="logits", seed=c["seed"],
                           logit_bias=bias, with_weights=False)
    ids = O.topk(wl.logits.numpy(), c["k"])
    local = ids[ids < c["n_local"]]
    return float(np.isin(local, order[:4]).mean()), int(local.size)


def main():
    lo, hi = 0.0, 2.0
    for _ in range(14):
        mid = 0.5 * (lo + hi)
        s, _ = share(mid)
        if s < 0.40:
            lo = mid
        else:
            hi = mid
    beta = round(0.5 * (lo + hi), 3)
    s, p = share(beta)
    res = {"beta": beta, "top4_share": s, "local_pairs": p,
           "note": "written by tests/golden/skew_beta.py (oracle top-k only)"}
    with open(os.path.join(os.path.dirname(__file__), "skew_beta.json"), "w") as f:
        json.dump(res, f, indent=1)
    print(res)


if __name__ == "__main__":
    torch.set_num_threads(8)
    main()
