"""Training-time relaxed forward of the controller and its regularisers.

TEST INFRASTRUCTURE (part of the CPU oracle): only tests, the smoke check and
the benchmark's CPU-baseline leg use it.  It shares no code with the GPU path.

Paper anchors (section / equation names of the TriRoute paper):
  * Sec. 3.6 per-axis whitening: each head reads its own detached whitening
    of the controller state, (h^ - mu^axis) / (sigma^axis + eps), with
    running statistics mu, sigma.
  * Sec. 3.4 heterogeneous relaxation: experts keep the top-k softmax of the
    inference router; the attention and bit decisions take the
    straight-through Gumbel-softmax, soft sample
    y~_o = softmax((z_o + g_o) / tau) with g ~ Gumbel(0, 1) i.i.d., forward
    value y = onehot(argmax_o y~_o).
  * Sec. 3.5 cost model: c^flops_t = sum_m y~^a_m kappa^a_m(t)
    + sum_{j in S_t} p-bar_j kappa^e, c^mem_t = sum_b y~^b_b 2 d_kv b,
    normalised by the dense cost of the same tokens.
  * Sec. 3.6 per-axis Switch balance loss L_bal = |O| sum_o f_o P_o, router
    z-loss L_z = mean_t (log sum_o exp z_o)^2, and the entropy floor
    L_ent = [zeta log |O| - H(p-bar)]_+.
  * Sec. 3.7 total loss (the regulariser part, the language-model loss
    aside) and projected dual ascent on an EMA of the normalised cost.
  * Algorithm 1 (one layer's training step): trunk, whitening, heads,
    ST-Gumbel / top-k, costs, losses; the dual update after the step.

Readings where the paper is silent or ambiguous (listed in the design notes):
  whitening acts on h^ = RMSNorm(h) gr, the input the heads read at
  inference, so frozen statistics fold into (W, c) (R18 there); the
  gradient-balance rescale changes only gradients, so the forward takes no
  rho; P_o and p-bar are means of the noise-free router probabilities
  softmax(z); f_o counts the hard (noisy) decisions; the attention axis
  counts (token, decision group) rows; the expert axis counts assignments,
  f_o = |{t : o in S_t}| / (k T); the null expert costs nothing; kappa^a is
  counted per head as in the hard accounting (R1, R31); C-bar is the ratio of
  the summed costs to the summed dense costs; the EMA is updated before the
  multiplier, and the regulariser uses the multipliers before the update.
"""
from __future__ import annotations

import numpy as np

from .layer import BITS, MODE_FULL, MODE_LOCAL, gelu, rmsnorm, softmax, _argmax_first

AXES = ("attention", "experts", "bits")


# ------------------------------------------------------------------ forward
def controller_state(L, tokens=None):
    """Sec. 3.3 trunk: n1 = Norm(x), u = GELU(W1 [n1; psi] + b1),
    h = W2 u + b2, h^ = RMSNorm(h; gr).  Returns (n1, h^)."""
    x = L["x"] if tokens is None else L["x"][tokens]
    psi = L["psi"] if tokens is None else L["psi"][tokens]
    n1 = rmsnorm(x, L["g1"])
    s = np.concatenate([n1, np.asarray(psi, np.float64)], axis=1)
    u = gelu(s @ np.asarray(L["W1"], np.float64).T + L["b1"])
    h = u @ np.asarray(L["W2"], np.float64).T + L["b2"]
    return n1, rmsnorm(h, L["gr"])


def whiten(hh, mu, sd, eps):
    """Sec. 3.6 whitening of one axis: (h^ - mu) / (sigma + eps), per feature."""
    return (np.asarray(hh, np.float64) - np.asarray(mu, np.float64)) / (
        np.asarray(sd, np.float64) + eps)


def relaxed_logits(L, R, tokens=None):
    """Head logits with each axis reading its whitened state.

    ``R["white_mu"]``, ``R["white_sd"]`` [3, d_r] (axis order attention,
    experts, bits) or None (no whitening).  Returns n1, h^, z^a [n, A, 3],
    z^e [n, E + 1], z^b [n, 4]."""
    cfg = L["cfg"]
    n1, hh = controller_state(L, tokens)
    if R.get("white_mu") is None:
        ha = he = hb = hh
    else:
        ha, he, hb = (whiten(hh, R["white_mu"][i], R["white_sd"][i], R["white_eps"])
                      for i in range(3))
    A = cfg.get("attn_groups") or cfg["H"]
    za = (ha @ np.asarray(L["Wa"], np.float64).T + L["ca"]).reshape(len(hh), A, 3)
    ze = he @ np.asarray(L["We"], np.float64).T + L["ce"]
    zb = hb @ np.asarray(L["Wb"], np.float64).T + L["cb"]
    return n1, hh, za, ze, zb


def st_gumbel(z, g, tau):
    """Sec. 3.4 ST-Gumbel forward over the last axis: the soft sample
    y~ = softmax((z + g) / tau) and the hard choice argmax y~ (first maximum).
    """
    assert tau > 0
    ys = softmax((np.asarray(z, np.float64) + np.asarray(g, np.float64)) / tau, axis=-1)
    flat = ys.reshape(-1, ys.shape[-1])
    y = np.array([_argmax_first(r) for r in flat], np.int64).reshape(ys.shape[:-1])
    return ys, y


def logsumexp(z):
    z = np.asarray(z, np.float64)
    m = np.max(z, axis=-1, keepdims=True)
    return (m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True)))[..., 0]


def topk_set(ze, k):
    """Sec. 3.2 (B) top-k of softmax(z^e): the k most probable options (lower
    id on ties), in ascending id."""
    p = softmax(ze, axis=-1)
    S = np.zeros((len(p), k), np.int64)
    for i in range(len(p)):
        order = sorted(range(p.shape[1]), key=lambda j: (-p[i, j], j))
        S[i] = sorted(order[:k])
    return S


def topk_gates(ze, S):
    """Renormalised weights p-bar_j = p_j / sum_{S_t} p (null included)."""
    p = softmax(ze, axis=-1)
    sel = np.take_along_axis(p, np.asarray(S, np.int64), axis=1)
    return sel / sel.sum(axis=1, keepdims=True)


# -------------------------------------------------------------------- costs
def relaxed_costs(cfg, ya, yb, S, gate, pos):
    """Sec. 3.5 per-token expected costs under the relaxed policy.

    ya [N, A, 3] attention soft samples (query head h reads group
    h // (H / A)), yb [N, 4], S [N, k] expert ids, gate [N, k] p-bar, pos [N]
    0-based positions.  kappa per head and key: 2 d_h multiply-accumulates
    (so a token whose H heads read t keys costs 2 d t), local reads
    min(P + 1, w) keys and full P + 1; kappa^e = 3 d d_f for a real expert,
    0 for the null; a token stored at width b adds 2 d_kv b bits.
    Returns c_flops, c_mem [N] and the dense costs of the same tokens
    (full attention in every head, one expert, 16-bit KV)."""
    H, dh, d, dff, w = cfg["H"], cfg["dh"], cfg["d"], cfg["d_ff"], cfg["w"]
    dkv = cfg["Hkv"] * dh
    A = ya.shape[1]
    t = np.asarray(pos, np.float64) + 1.0
    keys = {MODE_LOCAL: np.minimum(t, w), MODE_FULL: t}
    c_flops = np.zeros(len(t))
    for h in range(H):
        a = h // (H // A)
        for m, kt in keys.items():
            c_flops += ya[:, a, m] * 2.0 * dh * kt
    real = np.asarray(S) != 0
    c_flops += (np.where(real, gate, 0.0)).sum(axis=1) * 3.0 * d * dff
    c_mem = (np.asarray(yb, np.float64) * (2.0 * dkv * np.asarray(BITS, np.float64))).sum(axis=1)
    dense_flops = H * 2.0 * dh * t + 3.0 * d * dff
    dense_mem = np.full(len(t), 2.0 * dkv * 16)
    return c_flops, c_mem, dense_flops, dense_mem


# ------------------------------------------------------------------- losses
def entropy(p):
    p = np.asarray(p, np.float64)
    nz = p > 0
    return float(-(p[nz] * np.log(p[nz])).sum())


def axis_losses(f, P, lse, zeta):
    """Sec. 3.6 losses of one axis from its hard-decision fractions f_o,
    mean soft probabilities P_o (= p-bar) and the per-row log-sum-exp of the
    logits: L_bal = |O| sum f P, L_z = mean lse^2,
    L_ent = max(0, zeta log|O| - H(P))."""
    f = np.asarray(f, np.float64)
    P = np.asarray(P, np.float64)
    nO = len(f)
    Hp = entropy(P)
    return dict(lbal=float(nO * (f * P).sum()), lz=float(np.mean(np.asarray(lse) ** 2)),
                entropy=Hp, lent=max(0.0, zeta * np.log(nO) - Hp))


def usage(choice, n_opt, rows):
    """Fraction of ``rows`` hard choices taking each option."""
    c = np.bincount(np.asarray(choice, np.int64).reshape(-1), minlength=n_opt)
    return c / float(rows)


def relaxed_forward(L, R, forced=None):
    """Algorithm 1 steps 1-3, 5 and 6 (the regulariser part) for one layer.

    ``R``: g_attn [N, A, 3], g_bits [N, 4] Gumbel(0, 1) noise, tau_a, tau_b,
    white_mu / white_sd / white_eps, pos [N], zeta, alpha, beta, gamma,
    c_target (flops, mem), dual (lambda_flops, lambda_mem, ema_flops,
    ema_mem) or None, dual_lr, dual_ema.
    ``forced``: optional dict of hard decisions (ya_idx [N, A], yb_idx [N],
    S [N, k]) used in place of this side's argmax / top-k (the discretely
    forced comparison: soft values stay this side's own).
    """
    cfg = L["cfg"]
    H, k = cfg["H"], cfg["k"]
    n1, hh, za, ze, zb = relaxed_logits(L, R)
    N, A, _ = za.shape
    ya, ya_idx = st_gumbel(za, R["g_attn"], R["tau_a"])
    yb, yb_idx = st_gumbel(zb, R["g_bits"], R["tau_b"])
    S = topk_set(ze, k)
    if forced is not None:
        ya_idx, yb_idx, S = forced["ya_idx"], forced["yb_idx"], forced["S"]
    gate = topk_gates(ze, S)
    mode = np.repeat(np.asarray(ya_idx, np.uint8), H // A, axis=1)
    pa, pe, pb = softmax(za), softmax(ze), softmax(zb)
    c_flops, c_mem, d_flops, d_mem = relaxed_costs(cfg, ya, yb, S, gate, R["pos"])
    E1 = ze.shape[1]
    ax = {
        "attention": axis_losses(usage(ya_idx, 3, N * A), pa.reshape(-1, 3).mean(axis=0),
                                 logsumexp(za).reshape(-1), R["zeta"]),
        "experts": axis_losses(usage(S, E1, N * k), pe.mean(axis=0), logsumexp(ze), R["zeta"]),
        "bits": axis_losses(usage(yb_idx, 4, N), pb.mean(axis=0), logsumexp(zb), R["zeta"]),
    }
    ax["attention"].update(f=usage(ya_idx, 3, N * A), P=pa.reshape(-1, 3).mean(axis=0))
    ax["experts"].update(f=usage(S, E1, N * k), P=pe.mean(axis=0))
    ax["bits"].update(f=usage(yb_idx, 4, N), P=pb.mean(axis=0))
    cbar = np.array([c_flops.sum() / d_flops.sum(), c_mem.sum() / d_mem.sum()])
    dual = np.zeros(4) if R.get("dual") is None else np.asarray(R["dual"], np.float64)
    reg = regulariser(ax, cbar, dual[:2], R)
    out = dict(n1=n1, hh=hh, za=za, ze=ze, zb=zb, ya=ya, yb=yb, ya_idx=ya_idx, yb_idx=yb_idx,
               mode=mode, bit=np.asarray(yb_idx, np.uint8), S=S, gate=gate, pe=pe,
               c_flops=c_flops, c_mem=c_mem, dense_flops=d_flops, dense_mem=d_mem,
               cbar=cbar, axes=ax, reg=reg,
               h_mean=hh.mean(axis=0), h_var=hh.var(axis=0))
    if R.get("dual") is not None and R.get("dual_ema", 0.0) > 0.0:
        out["dual"] = dual_update(dual, cbar, R["c_target"], R["dual_lr"], R["dual_ema"])
    return out


def regulariser(ax, cbar, lam, R):
    """Sec. 3.7 total loss without L_LM: sum over the three axes of
    alpha L_bal + beta L_z + gamma L_ent, plus sum_r lambda_r (C-bar_r - C*_r)."""
    s = 0.0
    for a in AXES:
        s += R["alpha"] * ax[a]["lbal"] + R["beta"] * ax[a]["lz"] + R["gamma"] * ax[a]["lent"]
    for r in range(2):
        s += lam[r] * (cbar[r] - R["c_target"][r])
    return float(s)


def dual_update(dual, cbar, target, lr, m):
    """Sec. 3.7 projected dual ascent on an EMA of C-bar:
    ema <- (1 - m) ema + m C-bar, then lambda <- max(0, lambda + lr (ema - C*)).
    ``dual`` = (lambda_flops, lambda_mem, ema_flops, ema_mem)."""
    dual = np.asarray(dual, np.float64)
    ema = (1.0 - m) * dual[2:] + m * np.asarray(cbar, np.float64)
    lam = np.maximum(0.0, dual[:2] + lr * (ema - np.asarray(target, np.float64)))
    return np.concatenate([lam, ema])


def relaxed_margins(za, g_attn, tau_a, zb, g_bits, tau_b, ze, k):
    """Smallest gap that decides each token's relaxed choices: the top-2 gap
    of (z + g) / tau per attention group and for bits, and the k-th vs
    (k+1)-th expert logit gap."""
    def gap(v):
        s = np.sort(v, axis=-1)
        return s[..., -1] - s[..., -2]
    ga = gap((za + g_attn) / tau_a).min(axis=1)
    gb = gap((zb + g_bits) / tau_b)
    se = np.sort(ze, axis=-1)
    ge = se[:, -k] - se[:, -k - 1] if k < ze.shape[1] else np.full(len(ze), np.inf)
    return ga, gb, ge
