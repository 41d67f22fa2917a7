"""Pins of the relaxed (training-time) controller forward of the oracle.

Each pin checks the oracle against something other than itself: the
Gumbel-max sampling law, limits of the softmax temperature, library routines,
the inference router and the hard-decision cost accounting it must reduce to,
and closed forms of the losses and of the dual update.
"""
import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import gen
import oracle
from oracle import cost, relax
from oracle.ties import enforce_relaxed_margins


def _tiny(groups=None):
    L = gen.make_layer("tiny_f32_prefill", with_moe=False)
    if groups:
        L = gen.granularity_variant(L, groups)
    return L


def test_gumbel_max_law():
    """Sec. 3.4: argmax(z + g) with g ~ Gumbel(0, 1) is distributed as
    softmax(z), whatever tau > 0 (the temperature only shapes the soft
    sample).  A sign error on g or the wrong noise law fails this."""
    z = np.array([0.3, -1.1, 1.4, 0.0])
    n = 200_000
    g = gen.gumbel(7, "law", (n, 4)).astype(np.float64)
    p = scipy.special.softmax(z)
    for tau in (0.5, 1.0, 2.0):
        _, y = relax.st_gumbel(np.broadcast_to(z, (n, 4)), g, tau)
        freq = np.bincount(y, minlength=4) / n
        sd = np.sqrt(p * (1 - p) / n)
        assert np.all(np.abs(freq - p) < 5 * sd), (tau, freq, p)


def test_soft_sample_limits():
    z = gen.normal(3, "z", (50, 3)).astype(np.float64)
    g = gen.gumbel(3, "g", (50, 3)).astype(np.float64)
    # tau = 1 and no noise: the library softmax
    ys, _ = relax.st_gumbel(z, np.zeros_like(z), 1.0)
    np.testing.assert_allclose(ys, torch.softmax(torch.from_numpy(z), -1).numpy(), rtol=1e-12)
    # tau -> 0: the one-hot of argmax(z + g); tau -> inf: uniform
    ys, y = relax.st_gumbel(z, g, 1e-6)
    np.testing.assert_array_equal(y, np.argmax(z + g, axis=1))
    np.testing.assert_allclose(ys, np.eye(3)[y], atol=1e-12)
    ys, _ = relax.st_gumbel(z, g, 1e8)
    np.testing.assert_allclose(ys, 1 / 3, atol=1e-7)
    # temperature scales the log-odds: log(y~_i / y~_j) = (v_i - v_j) / tau
    ys, _ = relax.st_gumbel(z, g, 0.7)
    np.testing.assert_allclose(np.log(ys[:, 0] / ys[:, 1]), (z + g)[:, 0] / 0.7 - (z + g)[:, 1] / 0.7,
                               rtol=1e-10, atol=1e-10)


def test_whitening_identity_and_fold():
    """No whitening (mu = 0, sigma + eps = 1) gives the inference router's
    logits; general statistics equal the inference router with the affine
    map folded into the heads: W' = W diag(1 / (sigma + eps)),
    c' = c - W' mu."""
    L = _tiny()
    R = gen.relax_inputs(L)
    eps = R["white_eps"]
    ident = dict(R, white_mu=np.zeros((3, 128)), white_sd=np.full((3, 128), 1.0 - eps))
    _, _, za, ze, zb = relax.relaxed_logits(L, ident)
    _, za0, ze0, zb0 = oracle.router_logits(L)
    for a, b in ((za, za0), (ze, ze0), (zb, zb0)):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)
    F = dict(L)
    for i, (W, c) in enumerate((("Wa", "ca"), ("We", "ce"), ("Wb", "cb"))):
        Wp = np.asarray(L[W], np.float64) / (np.asarray(R["white_sd"][i], np.float64) + eps)
        F[W] = Wp
        F[c] = np.asarray(L[c], np.float64) - Wp @ np.asarray(R["white_mu"][i], np.float64)
    _, za1, ze1, zb1 = oracle.router_logits(F)
    _, _, za, ze, zb = relax.relaxed_logits(L, R)
    for a, b in ((za, za1), (ze, ze1), (zb, zb1)):
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-10)


def test_relaxed_experts_match_inference_topk():
    """Sec. 3.4: experts keep the inference top-k softmax (set and gates)."""
    L = _tiny()
    R = gen.relax_inputs(L, white=False)
    out = relax.relaxed_forward(L, R)
    _, za, ze, zb = oracle.router_logits(L)
    _, _, eidx, egate = oracle.decide(za, ze, zb, L["cfg"]["k"], L["cfg"]["H"])
    np.testing.assert_array_equal(out["S"], eidx)
    np.testing.assert_allclose(out["gate"], egate, rtol=1e-12)


@pytest.mark.parametrize("groups", [None, 2, 1])
def test_costs_reduce_to_hard_accounting(groups):
    """With one-hot soft samples the expected costs are the hard-decision
    accounting (Sec. 3.5 at tau -> 0, App. A; attention decisions broadcast
    over a decision group's heads); the expected cost is linear in the soft
    samples; the dense decisions cost exactly C-bar = 1."""
    L = _tiny(groups)
    cfg = L["cfg"]
    N, H, k = len(L["x"]), cfg["H"], cfg["k"]
    R = gen.relax_inputs(L)
    out = relax.relaxed_forward(L, R)
    ya1, yb1 = np.eye(3)[out["ya_idx"]], np.eye(4)[out["yb_idx"]]
    S = out["S"]
    cf, cm, df, dm = relax.relaxed_costs(cfg, ya1, yb1, S, np.ones_like(out["gate"]), R["pos"])
    mode = np.repeat(out["ya_idx"], H // out["za"].shape[1], axis=1)
    acc = cost.cost_terms(cfg, mode, out["bit"], S, R["pos"])
    assert cf.sum() == pytest.approx(acc["attn"] + acc["ffn"], rel=1e-13)
    assert cm.sum() == pytest.approx(acc["kv_bits"], rel=1e-13)
    dense = cost.dense_reference(cfg, R["pos"])
    assert df.sum() == pytest.approx(dense["attn"] + dense["ffn"], rel=1e-13)
    assert dm.sum() == pytest.approx(dense["kv_bits"], rel=1e-13)
    # dense decisions: full everywhere, 16 bits, one real expert with gate 1
    yaf = np.zeros((N, H, 3)); yaf[..., 2] = 1
    ybf = np.zeros((N, 4)); ybf[:, 3] = 1
    cf, cm, df, dm = relax.relaxed_costs(cfg, yaf, ybf, np.ones((N, 1), np.int64),
                                         np.ones((N, 1)), R["pos"])
    assert cf.sum() / df.sum() == pytest.approx(1.0, rel=1e-14)
    assert cm.sum() / dm.sum() == pytest.approx(1.0, rel=1e-14)
    # linearity in the soft samples
    lam = 0.3
    ya2, yb2 = np.roll(ya1, 1, axis=2), np.roll(yb1, 1, axis=1)
    c1 = relax.relaxed_costs(cfg, ya1, yb1, S, out["gate"], R["pos"])
    c2 = relax.relaxed_costs(cfg, ya2, yb2, S, out["gate"], R["pos"])
    cmix = relax.relaxed_costs(cfg, lam * ya1 + (1 - lam) * ya2, lam * yb1 + (1 - lam) * yb2, S,
                               out["gate"], R["pos"])
    for i in range(2):
        np.testing.assert_allclose(cmix[i], lam * c1[i] + (1 - lam) * c2[i], rtol=1e-12)
    # the null costs nothing: a set {null, e} costs kappa^e (1 - p-bar_null)
    Sn = np.tile(np.array([[0, 1]]), (N, 1))
    gn = np.tile(np.array([[0.25, 0.75]]), (N, 1))
    cf0, *_ = relax.relaxed_costs(cfg, np.zeros((N, H, 3)), yb1, Sn, gn, R["pos"])
    np.testing.assert_allclose(cf0, 0.75 * 3 * cfg["d"] * cfg["d_ff"], rtol=1e-14)
    assert k == 1


def test_balance_z_entropy_closed_forms():
    # balance: uniform usage gives 1, a collapse onto one option |O|, and
    # f = P gives |O| sum P^2 >= 1 (Cauchy-Schwarz) with equality iff uniform
    for n in (3, 4, 9):
        u = np.full(n, 1.0 / n)
        assert relax.axis_losses(u, u, np.zeros(2), 0.5)["lbal"] == pytest.approx(1.0)
        e = np.eye(n)[0]
        assert relax.axis_losses(e, e, np.zeros(2), 0.5)["lbal"] == pytest.approx(float(n))
        P = scipy.special.softmax(gen.normal(n, "p", (n,)).astype(np.float64))
        assert relax.axis_losses(P, P, np.zeros(2), 0.5)["lbal"] > 1.0
    # hard-decision fractions of a hand example
    np.testing.assert_allclose(relax.usage(np.array([0, 0, 1, 2]), 3, 4), [0.5, 0.25, 0.25])
    # z-loss of constant logits c: lse = c + log |O|
    z = np.full((5, 4), 1.7)
    lse = relax.logsumexp(z)
    np.testing.assert_allclose(lse, 1.7 + np.log(4), rtol=1e-14)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=1), rtol=1e-14)
    assert relax.axis_losses(np.eye(4)[0], np.eye(4)[0], lse, 0.5)["lz"] == pytest.approx(
        (1.7 + np.log(4)) ** 2)
    # entropy floor: inactive at uniform usage, zeta log|O| at a collapse,
    # the hinge value in between; H is the library entropy
    assert relax.axis_losses(np.full(3, 1 / 3), np.full(3, 1 / 3), lse, 0.5)["lent"] == 0.0
    assert relax.axis_losses(np.eye(3)[1], np.eye(3)[1], lse, 0.5)["lent"] == pytest.approx(
        0.5 * np.log(3))
    P = np.array([0.9, 0.05, 0.05])
    Hp = scipy.stats.entropy(P)
    assert relax.entropy(P) == pytest.approx(Hp, rel=1e-14)
    assert relax.axis_losses(P, P, lse, 0.7)["lent"] == pytest.approx(max(0, 0.7 * np.log(3) - Hp))


def test_dual_update_closed_form():
    d = np.array([0.3, 0.0, 0.5, 0.2])
    out = relax.dual_update(d, np.array([0.9, 0.1]), (0.5, 0.4), 0.05, 0.1)
    ema = np.array([0.9 * 0.5 + 0.1 * 0.9, 0.9 * 0.2 + 0.1 * 0.1])
    np.testing.assert_allclose(out[2:], ema)
    np.testing.assert_allclose(out[:2], [0.3 + 0.05 * (ema[0] - 0.5), 0.0])  # projected at 0
    # a constant cost drives the EMA to it geometrically and the price up
    # (over budget) without bound, or down to 0 (under budget)
    s = np.array([0.0, 1.0, 0.0, 0.0])
    for _ in range(400):
        s = relax.dual_update(s, np.array([0.8, 0.2]), (0.5, 0.4), 0.05, 0.1)
    np.testing.assert_allclose(s[2:], [0.8, 0.2], rtol=1e-12)
    assert s[0] > 5.0 and s[1] == 0.0


def test_regulariser_and_forward_consistency():
    """The regulariser is the weighted sum of the per-axis losses plus the
    priced budget violation; the forced forward with this side's own
    decisions reproduces the free one; the attention rows broadcast over a
    decision group."""
    for groups in (None, 2):
        L = _tiny(groups)
        R = gen.relax_inputs(L)
        enforce_relaxed_margins(L, R)
        out = relax.relaxed_forward(L, R)
        ax = out["axes"]
        want = sum(R["alpha"] * ax[a]["lbal"] + R["beta"] * ax[a]["lz"] + R["gamma"] * ax[a]["lent"]
                   for a in relax.AXES)
        want += 0.3 * (out["cbar"][0] - 0.5) + 0.7 * (out["cbar"][1] - 0.4)
        assert out["reg"] == pytest.approx(want, rel=1e-14)
        f = dict(ya_idx=out["ya_idx"], yb_idx=out["yb_idx"], S=out["S"])
        again = relax.relaxed_forward(L, R, forced=f)
        assert again["reg"] == out["reg"]
        H, A = L["cfg"]["H"], out["za"].shape[1]
        for h in range(H):
            np.testing.assert_array_equal(out["mode"][:, h], out["ya_idx"][:, h // (H // A)])
        assert np.all(out["cbar"] > 0) and np.all(out["cbar"] <= 1)
        for a in relax.AXES:
            assert ax[a]["f"].sum() == pytest.approx(1.0) and ax[a]["P"].sum() == pytest.approx(1.0)


def test_relaxed_margins_enforced():
    L = _tiny()
    R = gen.relax_inputs(L)
    enforce_relaxed_margins(L, R)
    _, _, za, ze, zb = relax.relaxed_logits(L, R)
    ga, gb, ge = relax.relaxed_margins(za, R["g_attn"], R["tau_a"], zb, R["g_bits"], R["tau_b"],
                                       ze, L["cfg"]["k"])
    assert min(ga.min(), gb.min(), ge.min()) >= 1e-4
