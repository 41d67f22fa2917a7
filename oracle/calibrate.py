"""Calibrate router head biases so hard decisions split as each workload asks.

TEST INFRASTRUCTURE (part of the CPU oracle).  Run as
``python -m oracle.calibrate`` from the repository root; it writes
``gen/router_bias.json``, which the seeded generator then reads.  The stored
biases are inputs (they shape the synthetic routing mix), not expected values.

Method: with the trunk fixed, logits are z = W h^ + c.  A fixed-point update
c <- c + (log target - log achieved) on the hard-decision fractions is run
per attention head (modes), on the bit head, and on the share of top-k
assignments per expert option, over a population of tokens drawn from the
workload's distribution.
"""
from __future__ import annotations

import json
import os
import sys

import numpy as np

import gen
from .layer import rmsnorm, gelu


def _trunk(L, x, psi):
    n1 = rmsnorm(x, L["g1"])
    s = np.concatenate([n1, np.asarray(psi, np.float64)], axis=1)
    u = gelu(s @ np.asarray(L["W1"], np.float64).T + L["b1"])
    h = u @ np.asarray(L["W2"], np.float64).T + L["b2"]
    return rmsnorm(h, L["gr"])


def _population(L, n_min=8192):
    cfg = L["cfg"]
    N = cfg["B"] * cfg["T"]
    if N >= 4096:
        return L["x"], L["psi"]
    x = gen.to_act(gen.normal(cfg["seed"], "calib_x", (n_min, cfg["d"])), cfg["act"])
    rel = L["psi"][:, 0]
    relp = np.resize(rel, n_min).astype(np.float32)
    psi = gen.token_psi(cfg["seed"] + 7919, n_min, relp)
    return x, psi


def _update(c, achieved, target, eta):
    live = target > 0
    c = c.copy()
    step = np.log(target[live]) - np.log(np.maximum(achieved[live], 1e-4))
    c[live] += eta * np.clip(step, -2.0, 2.0)
    c[~live] = -30.0
    return c


def calibrate(name, seed, iters=400, tol=0.004):
    L = gen.make_layer(name, seed, with_moe=False, biases={})
    cfg = L["cfg"]
    H, E, k = cfg["H"], cfg["E"], cfg["k"]
    x, psi = _population(L)
    hh = _trunk(L, x, psi)
    n = len(hh)
    base_a = (hh @ np.asarray(L["Wa"], np.float64).T).reshape(n, H, 3)
    base_e = hh @ np.asarray(L["We"], np.float64).T
    base_b = hh @ np.asarray(L["Wb"], np.float64).T
    t_mode = np.asarray(cfg["modes"], np.float64)
    t_bit = np.asarray(cfg["bits"], np.float64)
    t_exp = gen.expert_targets(cfg)
    ca = np.where(np.tile(t_mode, (H, 1)) > 0, 0.0, -30.0)
    cb = np.where(t_bit > 0, 0.0, -30.0)
    ce = np.where(t_exp > 0, 0.0, -30.0)
    # step size in units of the logits' spread across tokens
    spread = float(np.mean([base_a.std(axis=0).mean(), base_e.std(axis=0).mean(),
                            base_b.std(axis=0).mean()]))
    err = 1.0
    for it in range(iters):
        eta = spread * (0.5 if it < iters // 2 else 0.2)
        am = np.argmax(base_a + ca[None], axis=-1)                 # [n, H]
        fa = np.stack([(am == m).mean(axis=0) for m in range(3)], axis=1)
        ab = np.argmax(base_b + cb[None], axis=-1)
        fb = np.bincount(ab, minlength=4) / n
        ze = base_e + ce[None]
        top = np.argsort(-ze, axis=-1, kind="stable")[:, :k]
        fe = np.bincount(top.ravel(), minlength=E + 1) / (n * k)
        err = max(np.abs(fa - t_mode[None]).max(), np.abs(fb - t_bit).max(),
                  np.abs(fe - t_exp).max())
        if err < tol:
            break
        for h in range(H):
            ca[h] = _update(ca[h], fa[h], t_mode, eta)
        cb = _update(cb, fb, t_bit, eta)
        ce = _update(ce, fe, t_exp, eta)
    f32 = lambda a: [float(np.float32(v)) for v in np.ravel(a)]
    return dict(ca=f32(ca), ce=f32(ce), cb=f32(cb), err=float(err), pop=int(n))


def main(argv=None):
    out = {}
    for name, cfg in gen.CONFIGS.items():
        for seed in cfg["seeds"]:
            r = calibrate(name, seed)
            out[gen.bias_key(name, seed)] = r
            print(f"{name} seed {seed}: max fraction error {r['err']:.4f} "
                  f"over {r['pop']} tokens", flush=True)
    path = os.path.join(os.path.dirname(gen.__file__), "router_bias.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main(sys.argv[1:])
