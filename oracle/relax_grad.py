"""Backward pass of the relaxed controller forward (training time).

TEST INFRASTRUCTURE (part of the CPU oracle): only tests and the smoke check
use it.  It shares no code with the GPU path.

What is differentiated (Sec. 3.4-3.7, Algorithm 1 step 7 for the controller):
the soft outputs the rest of the layer consumes, y~^a and y~^b (the
straight-through estimator passes the language-model gradient of the hard
choice to the soft sample) and the expert gates p-bar, plus the regulariser
of Sec. 3.7 (balance, z and entropy-floor losses per axis and the priced
budget violation), with the hard choices, the usage fractions f_o, the
whitening statistics and the multipliers held constant (detached).  The
language-model part of each head's logit gradient is divided by that axis'
running gradient-balance factor rho (Sec. 3.4), which is then moved towards
the norm of that part: rho <- (1 - m) rho + m ||dL_LM / dz^axis||.

Chain, by hand, in the order of the forward: logits z (per axis) -> head
weights and biases, whitened h^ -> RMSNorm(h; gr) -> W2, b2 -> GELU ->
W1, b1 -> [Norm(x; g1); psi] -> g1, x, psi.

Readings (listed in the design notes): R42 the upstream inputs are
dL/dy~^a, dL/dy~^b and dL/dp-bar of the selected slots; R43 all three
heads' language-model gradients are balanced (attention, experts, bits),
rho's norm is the Frobenius norm over the batch of the unscaled gradient,
and the step uses rho before its update.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

from .layer import BITS, MODE_FULL, MODE_LOCAL, rmsnorm, softmax
from .relax import controller_state, whiten

EPS = 1e-6


def _softmax_rows_grad(p, g):
    """d/dz of sum(g * softmax(z)) for rows of softmax values p."""
    return p * (g - (p * g).sum(axis=-1, keepdims=True))


def _axis_reg_grad(p, f, lse, P, ent_active, alpha, beta, gamma, rows):
    """Gradient of alpha L_bal + beta L_z + gamma L_ent of one axis with
    respect to that axis' logits (p = softmax(z) per row, f held constant).
      L_bal = |O| sum_o f_o P_o,  P_o = mean over rows of p_o
      L_z   = mean over rows of lse^2
      L_ent = [zeta log|O| - H(P)]_+,  dH/dP_o = -(log P_o + 1)."""
    nO = p.shape[-1]
    g = alpha * nO / rows * _softmax_rows_grad(p, np.broadcast_to(f, p.shape))
    g = g + beta * 2.0 / rows * lse[..., None] * p
    if ent_active:
        logP = np.log(P)
        g = g + gamma / rows * _softmax_rows_grad(p, np.broadcast_to(logP + 1.0, p.shape))
    return g


def gelu_grad(y):
    y = np.asarray(y, np.float64)
    return 0.5 * (1.0 + erf(y / np.sqrt(2.0))) + y * np.exp(-0.5 * y * y) / np.sqrt(2.0 * np.pi)


def relaxed_backward(L, R, fwd, up, rho=(1.0, 1.0, 1.0), rho_m=0.0):
    """Gradients of the controller's parameters and inputs.

    ``fwd``: the output of ``relax.relaxed_forward`` (hard choices already
    taken); ``up``: g_ya [N, A, 3], g_yb [N, 4], g_gate [N, k], the
    language-model gradients of y~^a, y~^b and p-bar; ``rho``: the running
    gradient-balance factors (attention, experts, bits); ``rho_m``: their
    EMA momentum."""
    cfg = L["cfg"]
    H, dh, d, dff, w = cfg["H"], cfg["dh"], cfg["d"], cfg["d_ff"], cfg["w"]
    dkv = cfg["Hkv"] * dh
    za, ze, zb = fwd["za"], fwd["ze"], fwd["zb"]
    N, A, _ = za.shape
    k = fwd["S"].shape[1]
    E1 = ze.shape[1]
    ax = fwd["axes"]
    dual = np.zeros(4) if R.get("dual") is None else np.asarray(R["dual"], np.float64)
    lam_f, lam_m = dual[0], dual[1]
    Df, Dm = fwd["dense_flops"].sum(), fwd["dense_mem"].sum()
    zeta, alpha, beta, gamma = R["zeta"], R["alpha"], R["beta"], R["gamma"]

    def ent_active(a, nO):
        return zeta * np.log(nO) - ax[a]["entropy"] > 0

    # ---- attention logits: y~ = softmax((z + g) / tau_a)
    t = np.asarray(R["pos"], np.float64) + 1.0
    kap = np.zeros((N, 3))
    kap[:, MODE_LOCAL] = np.minimum(t, w)
    kap[:, MODE_FULL] = t
    kap *= (H // A) * 2.0 * dh
    ya = fwd["ya"]
    dza_lm = _softmax_rows_grad(ya, np.asarray(up["g_ya"], np.float64)) / R["tau_a"]
    dza_cost = _softmax_rows_grad(ya, np.broadcast_to((lam_f / Df) * kap[:, None, :], ya.shape)) / R["tau_a"]
    pa = softmax(za)
    from .relax import logsumexp
    dza_reg = _axis_reg_grad(pa, ax["attention"]["f"], logsumexp(za), ax["attention"]["P"],
                             ent_active("attention", 3), alpha, beta, gamma, N * A)
    # ---- bits: y~ = softmax((z + g) / tau_b), kappa^b = 2 d_kv b
    yb = fwd["yb"]
    dzb_lm = _softmax_rows_grad(yb, np.asarray(up["g_yb"], np.float64)) / R["tau_b"]
    kb = 2.0 * dkv * np.asarray(BITS, np.float64)
    dzb_cost = _softmax_rows_grad(yb, np.broadcast_to((lam_m / Dm) * kb, yb.shape)) / R["tau_b"]
    pb = softmax(zb)
    dzb_reg = _axis_reg_grad(pb, ax["bits"]["f"], logsumexp(zb), ax["bits"]["P"],
                             ent_active("bits", 4), alpha, beta, gamma, N)
    # ---- experts: p-bar_j = p_j / sum_S p over the selected set S
    S, gate = fwd["S"], fwd["gate"]
    Gp_lm = np.asarray(up["g_gate"], np.float64)
    Gp_cost = (lam_f / Df) * 3.0 * d * dff * (S != 0)
    dze_lm = np.zeros((N, E1))
    dze_cost = np.zeros((N, E1))
    sl_lm = _softmax_rows_grad(gate, Gp_lm)
    sl_cost = _softmax_rows_grad(gate, Gp_cost)
    for s in range(k):
        np.add.at(dze_lm, (np.arange(N), S[:, s]), sl_lm[:, s])
        np.add.at(dze_cost, (np.arange(N), S[:, s]), sl_cost[:, s])
    pe = fwd["pe"]
    dze_reg = _axis_reg_grad(pe, ax["experts"]["f"], logsumexp(ze), ax["experts"]["P"],
                             ent_active("experts", E1), alpha, beta, gamma, N)
    # ---- gradient balance
    lm = (dza_lm, dze_lm, dzb_lm)
    norms = np.array([np.sqrt((g * g).sum()) for g in lm])
    rho = np.asarray(rho, np.float64)
    dza = dza_lm / rho[0] + dza_cost + dza_reg
    dze = dze_lm / rho[1] + dze_cost + dze_reg
    dzb = dzb_lm / rho[2] + dzb_cost + dzb_reg
    rho_new = (1.0 - rho_m) * rho + rho_m * norms
    # ---- heads on the whitened state
    n1, hh = controller_state(L)
    if R.get("white_mu") is None:
        hw = [hh, hh, hh]
        inv = [np.ones(hh.shape[1])] * 3
    else:
        hw = [whiten(hh, R["white_mu"][i], R["white_sd"][i], R["white_eps"]) for i in range(3)]
        inv = [1.0 / (np.asarray(R["white_sd"][i], np.float64) + R["white_eps"]) for i in range(3)]
    dza2 = dza.reshape(N, 3 * A)
    out = dict(dza=dza, dze=dze, dzb=dzb, rho=rho_new, lm_norm=norms)
    out["dWa"], out["dca"] = dza2.T @ hw[0], dza2.sum(axis=0)
    out["dWe"], out["dce"] = dze.T @ hw[1], dze.sum(axis=0)
    out["dWb"], out["dcb"] = dzb.T @ hw[2], dzb.sum(axis=0)
    dhh = (dza2 @ np.asarray(L["Wa"], np.float64)) * inv[0] \
        + (dze @ np.asarray(L["We"], np.float64)) * inv[1] \
        + (dzb @ np.asarray(L["Wb"], np.float64)) * inv[2]
    # ---- trunk, recomputed in the forward's order
    x = np.asarray(L["x"], np.float64)
    psi = np.asarray(L["psi"], np.float64)
    s_in = np.concatenate([n1, psi], axis=1)
    a1 = s_in @ np.asarray(L["W1"], np.float64).T + L["b1"]
    u = 0.5 * a1 * (1.0 + erf(a1 / np.sqrt(2.0)))
    h = u @ np.asarray(L["W2"], np.float64).T + L["b2"]
    DR = h.shape[1]
    r = 1.0 / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + EPS)
    gr = np.asarray(L["gr"], np.float64)
    out["dgr"] = (dhh * h * r).sum(axis=0)
    gh = dhh * gr
    dh_ = r * gh - r ** 3 * h * (gh * h).sum(axis=1, keepdims=True) / DR
    out["dW2"], out["db2"] = dh_.T @ u, dh_.sum(axis=0)
    du = dh_ @ np.asarray(L["W2"], np.float64)
    da1 = du * gelu_grad(a1)
    out["dW1"], out["db1"] = da1.T @ s_in, da1.sum(axis=0)
    ds = da1 @ np.asarray(L["W1"], np.float64)
    dn1, out["dpsi"] = ds[:, :d], ds[:, d:]
    r1 = 1.0 / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + EPS)
    g1 = np.asarray(L["g1"], np.float64)
    out["dg1"] = (dn1 * x * r1).sum(axis=0)
    gx = dn1 * g1
    out["dx"] = r1 * gx - r1 ** 3 * x * (gx * x).sum(axis=1, keepdims=True) / d
    return out


def surrogate(L, R, forced, up):
    """The scalar whose gradient ``relaxed_backward`` returns at rho = 1:
    <g_ya, y~^a> + <g_yb, y~^b> + <g_gate, p-bar> + the regulariser, with the
    hard choices forced (for finite differences)."""
    from .relax import relaxed_forward
    f = relaxed_forward(L, R, forced=forced)
    return float((np.asarray(up["g_ya"]) * f["ya"]).sum() + (np.asarray(up["g_yb"]) * f["yb"]).sum()
                 + (np.asarray(up["g_gate"]) * f["gate"]).sum() + f["reg"])


__all__ = ["relaxed_backward", "surrogate", "gelu_grad", "rmsnorm"]
