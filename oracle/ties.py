"""Keep every routing decision of a synthetic layer away from a tie.

TEST INFRASTRUCTURE (part of the CPU oracle).  The GPU router computes its
logits in fp32 and the oracle in fp64; they differ by ~1e-6.  So that hard
decisions are well defined and can be compared bit for bit, any token whose
deciding logit gap (argmax per head, bit argmax, k-th vs (k+1)-th expert) is
below ``delta`` gets fresh psi_1..7 from the generator's per-token resample
stream until every gap clears ``delta``.
"""
from __future__ import annotations

import numpy as np

import gen
from .layer import router_logits, margins

DELTA = 1e-4


def enforce_margins(L, delta=DELTA, max_rounds=64):
    """Modify ``L['psi']`` in place; returns the number of resampled rows."""
    cfg = L["cfg"]
    _, za, ze, zb = router_logits(L)
    bad = np.flatnonzero(margins(za, ze, zb, cfg["k"]) < delta)
    attempt = np.zeros(len(L["x"]), np.int64)
    total = 0
    rounds = 0
    while len(bad) and rounds < max_rounds:
        for i in bad:
            L["psi"][i, 1:] = gen.resample_psi_row(cfg["seed"], int(i), int(attempt[i]))
            attempt[i] += 1
        total += len(bad)
        _, za, ze, zb = router_logits(L, bad)
        bad = bad[margins(za, ze, zb, cfg["k"]) < delta]
        rounds += 1
    if len(bad):
        raise RuntimeError(f"{len(bad)} tokens still within {delta} of a tie")
    return total
