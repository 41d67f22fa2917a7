"""Parity of the relaxed (training-time) controller forward against the oracle.

triroute_router_relaxed through the C ABI against ``oracle.relax`` on the same
seeded inputs: hard choices, top-k sets and the compaction bit exact (noise
and psi resampled off ties by the oracle's tie helper); logits, soft samples,
gates, expected costs and the batch statistics within the fp32 bound (the
controller is fp32 end to end on the GPU); the regulariser and the dual step
from the same statistics.  Shapes cover the one-wave tail (few tokens) and
the MFMA tail (many tokens), whitening on and off, and the three decision
granularities."""
import numpy as np
import pytest
import torch

import gen
import oracle
import paper_2607_06601_amd as tr
from oracle import relax
from oracle.ties import enforce_relaxed_margins
from paper_2607_06601_amd.device import DeviceLayer, to_dev

from _common import assert_close, err_ratio, layer, note, npy

pytestmark = pytest.mark.gpu
DEV = "cuda"
STAT_RTOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tr.lib()
    yield
    torch.cuda.synchronize()


def run_relaxed(L, R):
    cfg = L["cfg"]
    D = DeviceLayer(L, moe=False)
    c = D.cfg
    B, T, H, k, E = cfg["B"], cfg["T"], cfg["H"], cfg["k"], cfg["E"]
    A = cfg.get("attn_groups") or H
    N = B * T
    f32 = dict(dtype=torch.float32, device=DEV)
    t = dict(g_attn=to_dev(R["g_attn"], torch.float32), g_bits=to_dev(R["g_bits"], torch.float32),
             pos=to_dev(R["pos"], torch.int32))
    if R["white_mu"] is not None:
        t["mu"] = to_dev(R["white_mu"], torch.float32)
        t["sd"] = to_dev(R["white_sd"], torch.float32)
    t["dual"] = None if R.get("dual") is None else to_dev(np.asarray(R["dual"]), torch.float64)
    p = tr.RelaxParams(
        g_attn=t["g_attn"].data_ptr(), g_bits=t["g_bits"].data_ptr(), pos=t["pos"].data_ptr(),
        white_mu=t["mu"].data_ptr() if "mu" in t else None,
        white_sd=t["sd"].data_ptr() if "sd" in t else None, white_eps=R["white_eps"],
        tau_a=R["tau_a"], tau_b=R["tau_b"], zeta=R["zeta"], alpha=R["alpha"], beta=R["beta"],
        gamma=R["gamma"], dual=t["dual"].data_ptr() if t["dual"] is not None else None,
        dual_lr=R["dual_lr"], dual_ema=R["dual_ema"])
    p.c_target[0], p.c_target[1] = R["c_target"]
    o = dict(y_attn=torch.empty(N, A, 3, **f32), y_bits=torch.empty(N, 4, **f32),
             c_flops=torch.empty(N, **f32), c_mem=torch.empty(N, **f32),
             stats=torch.full((tr.RELAX_NSTAT,), float("nan"), dtype=torch.float64, device=DEV),
             p_exp=torch.empty(N, E + 1, **f32),
             usage_exp=torch.empty(2, E + 1, dtype=torch.float64, device=DEV),
             h_mean=torch.empty(128, **f32), h_var=torch.empty(128, **f32),
             z=torch.empty(N, 3 * A + E + 5, **f32))
    out = tr.RelaxOut(*(o[n].data_ptr() for n in (
        "y_attn", "y_bits", "c_flops", "c_mem", "stats", "p_exp", "usage_exp", "h_mean",
        "h_var", "z")))
    n1 = torch.empty(N, cfg["d"], dtype=D.act, device=DEV)
    mode = torch.empty(N, H, dtype=torch.uint8, device=DEV)
    bit = torch.empty(N, dtype=torch.uint8, device=DEV)
    eidx = torch.empty(N, k, dtype=torch.int32, device=DEV)
    egate = torch.empty(N, k, **f32)
    cmp = tr.CompactionBuffers(c, B, T)
    ws = tr.workspace(c, tr.OP_ROUTER_RELAXED, B, T)
    tr.router_relaxed(c, B, T, D.x, D.psi, D.rw, p, n1, mode, bit, eidx, egate, cmp.struct, out,
                      ws)
    torch.cuda.synchronize()
    o.update(mode=mode, bit=bit, eidx=eidx, egate=egate, cmp=cmp, dual=t["dual"])
    return {n: (npy(v) if isinstance(v, torch.Tensor) else v) for n, v in o.items()}


def _scalar(gpu, ref, name):
    err = abs(gpu - ref)
    bound = STAT_RTOL * abs(ref) + 1e-9
    note(name, err / bound)
    assert err <= bound, f"{name}: gpu {gpu!r} ref {ref!r}"


CASES = [  # (workload, attention decision groups, whitening, dual state)
    ("tiny_f32_prefill", None, True, True),
    ("160m_bf16_prefill", None, True, True),
    ("1p3b_bf16_prefill", 1, False, False),
    ("1p3b_bf16_decode", 4, True, True),
    ("410m_bf16_decode", None, False, True),
]


@pytest.mark.parametrize("name,groups,white,dual", CASES)
def test_relaxed_forward_matches_oracle(name, groups, white, dual):
    L = layer(name, moe=False)
    if groups is not None:
        L = gen.granularity_variant(L, groups)
    cfg = L["cfg"]
    B, T, H, E, k = cfg["B"], cfg["T"], cfg["H"], cfg["E"], cfg["k"]
    R = gen.relax_inputs(L, white=white)
    if not dual:
        R["dual"] = None
    enforce_relaxed_margins(L, R)
    print(f"relaxed forward {name} groups={groups} white={white} N={B * T}", flush=True)
    g = run_relaxed(L, R)
    ref = relax.relaxed_forward(L, R)
    # hard choices, sets and gates
    np.testing.assert_array_equal(g["mode"], ref["mode"])
    np.testing.assert_array_equal(g["bit"], ref["bit"])
    np.testing.assert_array_equal(g["eidx"], ref["S"])
    np.testing.assert_allclose(g["egate"], ref["gate"], rtol=2e-5, atol=1e-6)
    # logits (whitened) and the soft values
    A = ref["za"].shape[1]
    z_ref = np.concatenate([ref["za"].reshape(len(ref["za"]), -1), ref["ze"], ref["zb"]], axis=1)
    assert_close(g["z"], z_ref, "f32", "z (whitened logits)")
    assert_close(g["y_attn"], ref["ya"], "f32", "y~ attention")
    assert_close(g["y_bits"], ref["yb"], "f32", "y~ bits")
    assert_close(g["p_exp"], ref["pe"], "f32", "softmax z^e")
    assert_close(g["c_flops"], ref["c_flops"], "f32", "c_flops")
    assert_close(g["c_mem"], ref["c_mem"], "f32", "c_mem")
    # batch statistics and losses
    st = g["stats"]
    for i, a in enumerate(relax.AXES):
        ax = ref["axes"][a]
        _scalar(st[tr.RS_LBAL + i], ax["lbal"], f"L_bal {a}")
        _scalar(st[tr.RS_LZ + i], ax["lz"], f"L_z {a}")
        _scalar(st[tr.RS_LENT + i], ax["lent"], f"L_ent {a}")
        _scalar(st[tr.RS_ENTROPY + i], ax["entropy"], f"H {a}")
    np.testing.assert_array_equal(st[tr.RS_F_ATTN:tr.RS_F_ATTN + 3], ref["axes"]["attention"]["f"])
    np.testing.assert_array_equal(st[tr.RS_F_BITS:tr.RS_F_BITS + 4], ref["axes"]["bits"]["f"])
    np.testing.assert_array_equal(g["usage_exp"][0], ref["axes"]["experts"]["f"])
    np.testing.assert_allclose(st[tr.RS_P_ATTN:tr.RS_P_ATTN + 3], ref["axes"]["attention"]["P"],
                               rtol=STAT_RTOL, atol=1e-9)
    np.testing.assert_allclose(st[tr.RS_P_BITS:tr.RS_P_BITS + 4], ref["axes"]["bits"]["P"],
                               rtol=STAT_RTOL, atol=1e-9)
    np.testing.assert_allclose(g["usage_exp"][1], ref["axes"]["experts"]["P"], rtol=STAT_RTOL,
                               atol=1e-9)
    for r, rn in enumerate(("flops", "mem")):
        _scalar(st[tr.RS_CBAR + r], ref["cbar"][r], f"C-bar {rn}")
        _scalar(st[tr.RS_COST + r], (ref["c_flops"], ref["c_mem"])[r].sum(), f"cost {rn}")
        _scalar(st[tr.RS_DENSE + r], (ref["dense_flops"], ref["dense_mem"])[r].sum(),
                f"dense {rn}")
    _scalar(st[tr.RS_REG], ref["reg"], "regulariser")
    assert_close(g["h_mean"], ref["h_mean"], "f32", "mean h^")
    assert_close(g["h_var"], ref["h_var"], "f32", "var h^")
    if dual:
        np.testing.assert_allclose(g["dual"], ref["dual"], rtol=STAT_RTOL, atol=1e-9)
    # compaction of the relaxed decisions
    cm = oracle.compact(ref["mode"], ref["S"].astype(np.int32), B, T, H, E, k)
    cnt = g["cmp"].attn_cnt.cpu().numpy()
    np.testing.assert_array_equal(cnt, cm["attn_cnt"])
    idx = g["cmp"].attn_idx.cpu().numpy().reshape(B * H * 2, T)
    for s in range(B * H * 2):
        np.testing.assert_array_equal(idx[s, :cnt[s]], cm["attn_idx"][s, :cnt[s]])
    np.testing.assert_array_equal(g["cmp"].exp_cnt.cpu().numpy(), cm["exp_cnt"])
    nreal = int(cm["exp_off"][-1])
    np.testing.assert_array_equal(g["cmp"].exp_rows.cpu().numpy()[:nreal], cm["exp_rows"])


def test_relaxed_forward_is_deterministic_and_noise_free_limit():
    """Two calls give bit-identical statistics (fixed-order reductions); with
    zero noise and no whitening the hard choices are the inference router's."""
    L = layer("160m_bf16_prefill", moe=False)
    R = gen.relax_inputs(L, white=False)
    R["g_attn"][:] = 0
    R["g_bits"][:] = 0
    R["dual"] = None
    a = run_relaxed(L, R)
    b = run_relaxed(L, R)
    np.testing.assert_array_equal(a["stats"], b["stats"])
    np.testing.assert_array_equal(a["usage_exp"], b["usage_exp"])
    np.testing.assert_array_equal(a["h_var"], b["h_var"])
    _, za, ze, zb = oracle.router_logits(L)
    mode, bit, eidx, _ = oracle.decide(za, ze, zb, L["cfg"]["k"], L["cfg"]["H"])
    np.testing.assert_array_equal(a["mode"], mode)
    np.testing.assert_array_equal(a["bit"], bit)
    np.testing.assert_array_equal(a["eidx"], eidx)


# ------------------------------------------------------------------ backward
from oracle import relax_grad  # noqa: E402

GRAD_KEYS = [("dW1", "W1"), ("db1", "b1"), ("dW2", "W2"), ("db2", "b2"), ("dgr", "gr"),
             ("dWa", "Wa"), ("dca", "ca"), ("dWe", "We"), ("dce", "ce"), ("dWb", "Wb"),
             ("dcb", "cb"), ("dg1", "g1")]


def run_relaxed_backward(L, R, g, up, rho, rho_m):
    cfg = L["cfg"]
    D = DeviceLayer(L, moe=False)
    c = D.cfg
    B, T = cfg["B"], cfg["T"]
    N = B * T
    f32 = dict(dtype=torch.float32, device=DEV)
    t = dict(pos=to_dev(R["pos"], torch.int32))
    if R["white_mu"] is not None:
        t["mu"] = to_dev(R["white_mu"], torch.float32)
        t["sd"] = to_dev(R["white_sd"], torch.float32)
    p = tr.RelaxParams(pos=t["pos"].data_ptr(), white_mu=t["mu"].data_ptr() if "mu" in t else None,
                       white_sd=t["sd"].data_ptr() if "sd" in t else None,
                       white_eps=R["white_eps"], tau_a=R["tau_a"], tau_b=R["tau_b"],
                       zeta=R["zeta"], alpha=R["alpha"], beta=R["beta"], gamma=R["gamma"])
    fw = {n: to_dev(g[n], torch.float32) for n in ("y_attn", "y_bits")}
    fw["stats"] = to_dev(g["stats"], torch.float64)
    fw["usage_exp"] = to_dev(g["usage_exp"], torch.float64)
    fwd = tr.RelaxOut(y_attn=fw["y_attn"].data_ptr(), y_bits=fw["y_bits"].data_ptr(),
                      stats=fw["stats"].data_ptr(), usage_exp=fw["usage_exp"].data_ptr())
    eidx = to_dev(g["eidx"], torch.int32)
    egate = to_dev(g["egate"], torch.float32)
    u = {n: to_dev(up[n], torch.float32) for n in ("g_ya", "g_yb", "g_gate")}
    lam = None if R.get("dual") is None else to_dev(np.asarray(R["dual"][:2]), torch.float64)
    rho_t = to_dev(np.asarray(rho, np.float64), torch.float64)
    gin = tr.RelaxGradIn(g_attn=u["g_ya"].data_ptr(), g_bits=u["g_yb"].data_ptr(),
                         g_gate=u["g_gate"].data_ptr(), lambda_=lam.data_ptr() if lam is not None else None,
                         rho=rho_t.data_ptr(), rho_m=rho_m)
    out = {n: torch.full(np.shape(L[w]), float("nan"), **f32) for n, w in GRAD_KEYS}
    out["dx"] = torch.full((N, cfg["d"]), float("nan"), **f32)
    out["dpsi"] = torch.full((N, 8), float("nan"), **f32)
    out["lm_norm"] = torch.zeros(3, dtype=torch.float64, device=DEV)
    go = tr.RelaxGradOut(**{n: v.data_ptr() for n, v in out.items()})
    ws = tr.workspace(c, tr.OP_ROUTER_RELAXED_BACKWARD, B, T)
    tr.router_relaxed_backward(c, B, T, D.x, D.psi, D.rw, p, fwd, eidx, egate, gin, go, ws)
    torch.cuda.synchronize()
    res = {n: npy(v) for n, v in out.items()}
    res["rho"] = npy(rho_t)
    return res


BWD_CASES = [  # (workload, groups, whitening, k override, zeta)
    ("tiny_f32_prefill", None, True, 2, 0.5),
    ("160m_bf16_prefill", None, True, None, 1.0),
    ("1p3b_bf16_decode", 4, False, None, 0.5),
]


@pytest.mark.parametrize("name,groups,white,k,zeta", BWD_CASES)
def test_relaxed_backward_matches_oracle(name, groups, white, k, zeta):
    L = layer(name, moe=False)
    if k is not None:
        L["cfg"] = dict(L["cfg"], k=k)
    if groups is not None:
        L = gen.granularity_variant(L, groups)
    R = gen.relax_inputs(L, white=white)
    R["zeta"] = zeta
    enforce_relaxed_margins(L, R)
    print(f"relaxed backward {name} groups={groups} white={white} k={L['cfg']['k']}", flush=True)
    g = run_relaxed(L, R)
    ref = relax.relaxed_forward(L, R)
    np.testing.assert_array_equal(g["eidx"], ref["S"])
    N, A = ref["za"].shape[:2]
    kk = L["cfg"]["k"]
    up = dict(g_ya=gen.normal(9, "bwd_ga", (N, A, 3)), g_yb=gen.normal(9, "bwd_gb", (N, 4)),
              g_gate=gen.normal(9, "bwd_gg", (N, kk)))
    rho, rho_m = (1.5, 0.8, 2.5), 0.1
    gb = run_relaxed_backward(L, R, g, up, rho, rho_m)
    want = relax_grad.relaxed_backward(L, R, ref, {n: np.asarray(v, np.float64) for n, v in up.items()},
                                       rho=rho, rho_m=rho_m)
    names = [n for n, _ in GRAD_KEYS] + ["dx", "dpsi"]
    for n in names:  # every ratio first, so that one failure shows them all
        print(f"  {n}: max err/bound {err_ratio(gb[n], want[n], 'f32') / GRAD_FACTOR:.3f}", flush=True)
    for n in names:
        assert_close(gb[n], want[n], "f32", n, factor=GRAD_FACTOR)
    np.testing.assert_allclose(gb["lm_norm"], want["lm_norm"], rtol=1e-4)
    np.testing.assert_allclose(gb["rho"], want["rho"], rtol=1e-4)


# fp32 gradients summed over up to 16384 tokens in chunks of 128 (fp32 within
# a chunk, fp64 across): the tolerance is the fp32 bound times this factor
GRAD_FACTOR = 1.0
