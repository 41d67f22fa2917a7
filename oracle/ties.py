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


def enforce_relaxed_margins(L, R, delta=DELTA, max_rounds=64):
    """The relaxed forward's counterpart: a token whose ST-Gumbel choice
    (top-2 gap of (z + g) / tau per attention group or for bits) is within
    ``delta`` of a tie gets fresh noise rows from the generator's resample
    stream; one whose expert top-k (on the whitened logits) is gets fresh
    psi_1..7.  Modifies ``R['g_attn']``, ``R['g_bits']`` and ``L['psi']`` in
    place; returns the number of resampled rows."""
    from .relax import relaxed_logits, relaxed_margins
    cfg = L["cfg"]
    seed, k = cfg["seed"], cfg["k"]
    attempt = np.zeros(len(L["x"]), np.int64)
    total = 0
    rows = np.arange(len(L["x"]))
    for _ in range(max_rounds):
        _, _, za, ze, zb = relaxed_logits(L, R, rows)
        ga, gb, ge = relaxed_margins(za, R["g_attn"][rows], R["tau_a"], zb, R["g_bits"][rows],
                                     R["tau_b"], ze, k)
        bad_g = rows[(ga < delta) | (gb < delta)]
        bad_e = rows[ge < delta]
        if not len(bad_g) and not len(bad_e):
            return total
        for i in bad_g:
            R["g_attn"][i] = gen.resample_gumbel_row(seed, "g_attn", int(i), int(attempt[i]),
                                                     R["g_attn"].shape[1:])
            R["g_bits"][i] = gen.resample_gumbel_row(seed, "g_bits", int(i), int(attempt[i]), 4)
        for i in bad_e:
            L["psi"][i, 1:] = gen.resample_psi_row(seed, int(i), 1000 + int(attempt[i]))
        bad = np.union1d(bad_g, bad_e)
        attempt[bad] += 1
        total += len(bad)
        rows = bad
    raise RuntimeError(f"{len(rows)} tokens still within {delta} of a relaxed tie")
