"""Pins of the relaxed controller's backward pass (oracle).

The hand-derived gradients are checked against central finite differences
of the scalar they differentiate (the upstream-weighted soft outputs plus the
regulariser, hard choices held), for every kind of parameter and input, with
the entropy floor inactive and active, per-head and grouped attention
decisions, and top-2 experts (so the gate path is live); the gradient-balance
scaling and its update are checked against their closed forms.
"""
import numpy as np
import pytest

import gen
from oracle import relax, relax_grad
from oracle.ties import enforce_relaxed_margins


def _setup(groups=None, k=2, zeta=0.5, white=True):
    L = gen.make_layer("tiny_f32_prefill", with_moe=False)
    L["cfg"] = dict(L["cfg"], k=k)
    if groups:
        L = gen.granularity_variant(L, groups)
    R = gen.relax_inputs(L, white=white)
    R["zeta"] = zeta
    enforce_relaxed_margins(L, R)
    # parameters in fp64 so that finite differences see the exact function
    for n in ("x", "psi", "g1", "W1", "b1", "W2", "b2", "gr", "Wa", "ca", "We", "ce", "Wb", "cb"):
        L[n] = np.array(L[n], np.float64)
    fwd = relax.relaxed_forward(L, R)
    N, A = fwd["za"].shape[:2]
    up = dict(g_ya=gen.normal(5, "up_a", (N, A, 3)).astype(np.float64),
              g_yb=gen.normal(5, "up_b", (N, 4)).astype(np.float64),
              g_gate=gen.normal(5, "up_g", (N, k)).astype(np.float64))
    forced = dict(ya_idx=fwd["ya_idx"], yb_idx=fwd["yb_idx"], S=fwd["S"])
    return L, R, fwd, up, forced


# (parameter, gradient key)
PARAMS = [("W1", "dW1"), ("b1", "db1"), ("W2", "dW2"), ("b2", "db2"), ("gr", "dgr"),
          ("Wa", "dWa"), ("ca", "dca"), ("We", "dWe"), ("ce", "dce"), ("Wb", "dWb"),
          ("cb", "dcb"), ("g1", "dg1"), ("x", "dx"), ("psi", "dpsi")]


@pytest.mark.parametrize("groups,zeta,white", [(None, 0.5, True), (2, 1.0, True),
                                               (None, 1.0, False)])
def test_gradients_match_finite_differences(groups, zeta, white):
    L, R, fwd, up, forced = _setup(groups, zeta=zeta, white=white)
    g = relax_grad.relaxed_backward(L, R, fwd, up)
    if zeta == 1.0:  # the entropy floor acts on every axis (H(P) < log |O|)
        assert all(fwd["axes"][a]["lent"] > 0 for a in relax.AXES)
    rng = np.random.default_rng(11)
    for name, key in PARAMS:
        P = L[name]
        G = g[key]
        assert G.shape == P.shape, (name, G.shape, P.shape)
        flat = P.reshape(-1)
        idx = rng.choice(flat.size, size=min(6, flat.size), replace=False)
        for i in idx:
            h = 1e-6 * max(1.0, abs(flat[i]))
            old = flat[i]
            flat[i] = old + h
            jp = relax_grad.surrogate(L, R, forced, up)
            flat[i] = old - h
            jm = relax_grad.surrogate(L, R, forced, up)
            flat[i] = old
            fd = (jp - jm) / (2 * h)
            an = G.reshape(-1)[i]
            assert abs(fd - an) <= 1e-5 * max(1.0, abs(fd)), (name, i, fd, an)


def test_gradient_balance_scaling_and_update():
    """The language-model part of each axis' logit gradient is divided by
    that axis' rho; rho moves by (1 - m) rho + m ||that part||."""
    L, R, fwd, up, _ = _setup()
    R["dual"] = None  # no budget term: the remaining regulariser part does not scale
    g1 = relax_grad.relaxed_backward(L, R, fwd, up)
    zero = {k: np.zeros_like(v) for k, v in up.items()}
    g0 = relax_grad.relaxed_backward(L, R, fwd, zero)
    rho = (2.0, 0.5, 4.0)
    gs = relax_grad.relaxed_backward(L, R, fwd, up, rho=rho, rho_m=0.25)
    for i, key in enumerate(("dza", "dze", "dzb")):
        lm = g1[key] - g0[key]
        np.testing.assert_allclose(gs[key], g0[key] + lm / rho[i], rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(gs["lm_norm"][i], np.sqrt((lm * lm).sum()), rtol=1e-12)
        assert gs["rho"][i] == pytest.approx(0.75 * rho[i] + 0.25 * gs["lm_norm"][i])
    assert np.all(g0["lm_norm"] == 0)


def test_gelu_derivative():
    from oracle.layer import gelu
    y = np.linspace(-6, 6, 121)
    h = 1e-6
    fd = (gelu(y + h) - gelu(y - h)) / (2 * h)
    np.testing.assert_allclose(relax_grad.gelu_grad(y), fd, rtol=1e-7, atol=1e-9)
