"""Seeded synthetic inputs for one TriRoute-routed layer.

This module only draws numbers: shapes, value distributions and routing
mixes of the five workloads (160M-1.3B-class layers, Table 2 shapes).  It holds
none of the layer's arithmetic, so both the CPU oracle and the GPU path can
take their inputs from here.

Every tensor is drawn from its own PCG64 stream keyed by (seed, tensor name,
optional index), so the draw order never changes a value.  Values are drawn in
fp32 and rounded once (round-to-nearest-even) to the activation dtype; both
sides receive exactly those values.

Router head biases are not drawn: they are the per-workload calibrated values
stored in ``router_bias.json`` (written by the oracle's calibration script),
so that the hard decisions split as each workload asks.
"""
from __future__ import annotations

import json
import os
import zlib

import numpy as np

BITS = (2, 4, 8, 16)
MODES = ("skip", "local", "full")
D_PSI = 8
D_ROUTER = 128

# Workload table.  Fractions are listed in the order of the enumerations:
# modes (skip, local, full), bit widths (2, 4, 8, 16).  ``experts`` is the
# target share of top-k assignments over the E+1 options (index 0 = null).
CONFIGS = {
    "tiny_f32_prefill": dict(
        kind="prefill", B=1, T=128, d=256, H=4, Hkv=1, dh=64, w=32, E=4, k=1,
        d_ff=512, G=32, act="f32", seeds=(0,),
        modes=(0.30, 0.40, 0.30), bits=(0.25, 0.25, 0.25, 0.25),
        experts="uniform"),
    "160m_bf16_prefill": dict(
        kind="prefill", B=8, T=2048, d=768, H=12, Hkv=3, dh=64, w=128, E=8,
        k=2, d_ff=2048, G=64, act="bf16", seeds=(1, 2, 3),
        modes=(0.25, 0.45, 0.30), bits=(0.15, 0.35, 0.35, 0.15),
        experts="uniform"),
    "410m_bf16_decode": dict(
        kind="decode", B=64, T=1, ctx=8192, d=1024, H=16, Hkv=4, dh=64, w=256,
        E=8, k=2, d_ff=2816, G=64, act="bf16", seeds=(103,),
        modes=(0.25, 0.45, 0.30), bits=(0.20, 0.40, 0.30, 0.10),
        ctx_bits=(0.20, 0.40, 0.30, 0.10), experts="uniform"),
    "1p3b_bf16_prefill": dict(
        kind="prefill", B=4, T=4096, d=2048, H=16, Hkv=4, dh=128, w=512, E=16,
        k=2, d_ff=5632, G=64, act="bf16", seeds=(104,),
        modes=(0.20, 0.50, 0.30), bits=(0.15, 0.35, 0.35, 0.15),
        experts="uniform"),
    "1p3b_bf16_decode": dict(
        kind="decode", B=32, T=1, ctx=32768, d=2048, H=16, Hkv=4, dh=128,
        w=1024, E=16, k=2, d_ff=5632, G=64, act="bf16", seeds=(105,),
        modes=(0.20, 0.50, 0.30), bits=(0.70, 0.20, 0.0, 0.10),
        ctx_bits=(0.70, 0.20, 0.0, 0.10), experts="skewed"),
}

_BIAS_FILE = os.path.join(os.path.dirname(__file__), "router_bias.json")


def expert_targets(cfg: dict) -> np.ndarray:
    """Target share of assignments per option 0..E (0 = null)."""
    E = cfg["E"]
    if cfg["experts"] == "uniform":
        return np.full(E + 1, 1.0 / (E + 1))
    if cfg["experts"] == "skewed":
        # two hot experts take 30% each, the null 15%, the rest share 25%
        t = np.full(E + 1, 0.25 / (E - 2))
        t[0], t[1], t[2] = 0.15, 0.30, 0.30
        return t
    raise ValueError(cfg["experts"])


def stream(seed: int, name: str, *index: int) -> np.random.Generator:
    key = [int(seed), zlib.crc32(name.encode())] + [int(i) for i in index]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def to_act(a: np.ndarray, act: str) -> np.ndarray:
    if act == "bf16":
        return round_bf16(a)
    if act == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    if act == "f64":
        return np.ascontiguousarray(a, dtype=np.float64)
    raise ValueError(act)


def normal(seed, name, shape, std=1.0, *index):
    g = stream(seed, name, *index)
    return (g.standard_normal(shape, dtype=np.float32) * np.float32(std))


def load_biases() -> dict:
    if not os.path.exists(_BIAS_FILE):
        return {}
    with open(_BIAS_FILE) as f:
        return json.load(f)


def bias_key(name: str, seed: int) -> str:
    return f"{name}/seed{seed}"


def token_psi(seed: int, n_tok: int, rel_pos: np.ndarray) -> np.ndarray:
    """Side features: psi_0 = relative position, psi_1..7 ~ N(0, 1)."""
    psi = np.empty((n_tok, D_PSI), np.float32)
    psi[:, 0] = rel_pos
    psi[:, 1:] = normal(seed, "psi", (n_tok, D_PSI - 1))
    return psi


def resample_psi_row(seed: int, token: int, attempt: int) -> np.ndarray:
    """Fresh psi_1..7 for one token (used to move a token off a routing tie)."""
    return stream(seed, "psi_resample", token, attempt).standard_normal(
        D_PSI - 1, dtype=np.float32)


def make_layer(name: str, seed: int | None = None, *, act: str | None = None,
               with_moe: bool = True, biases: dict | None = None) -> dict:
    """Draw every input of one routed layer for workload ``name``.

    Returns a dict with ``cfg`` (shape fields plus ``name``/``seed``/``act``),
    the activations ``x`` [N, d] and ``psi`` [N, 8], fp32 router weights, the
    act-dtype attention / expert weights, and per-token positions.
    """
    cfg = dict(CONFIGS[name])
    seed = cfg["seeds"][0] if seed is None else seed
    act = act or cfg["act"]
    cfg.update(name=name, seed=seed, act=act)
    B, T, d, H, Hkv, dh = (cfg[k] for k in ("B", "T", "d", "H", "Hkv", "dh"))
    E, dff = cfg["E"], cfg["d_ff"]
    N = B * T
    L = {"cfg": cfg}
    L["x"] = to_act(normal(seed, "x", (N, d)), act)
    if cfg["kind"] == "prefill":
        rel = np.tile(np.arange(T, dtype=np.float32) / np.float32(T), B)
    else:
        ctx = cfg["ctx"]
        rel = np.full(N, np.float32(ctx) / np.float32(ctx + 1), np.float32)
    L["psi"] = token_psi(seed, N, rel)
    # router (fp32 end to end); whitening and the gradient-balance scale are
    # already folded into the head weights and biases
    dr = D_ROUTER
    L["g1"] = to_act(1.0 + normal(seed, "g1", (d,), 0.02), act)
    L["W1"] = normal(seed, "W1", (dr, d + D_PSI), 0.02)
    L["b1"] = normal(seed, "b1", (dr,), 0.02)
    L["W2"] = normal(seed, "W2", (dr, dr), 0.02)
    L["b2"] = normal(seed, "b2", (dr,), 0.02)
    L["gr"] = 1.0 + normal(seed, "gr", (dr,), 0.02)
    L["Wa"] = normal(seed, "Wa", (3 * H, dr), 0.02)
    L["We"] = normal(seed, "We", (E + 1, dr), 0.02)
    L["Wb"] = normal(seed, "Wb", (4, dr), 0.02)
    biases = load_biases() if biases is None else biases
    bk = biases.get(bias_key(name, seed))
    if bk is not None:
        L["ca"] = np.asarray(bk["ca"], np.float32)
        L["ce"] = np.asarray(bk["ce"], np.float32)
        L["cb"] = np.asarray(bk["cb"], np.float32)
    else:
        L["ca"] = np.zeros(3 * H, np.float32)
        L["ce"] = np.zeros(E + 1, np.float32)
        L["cb"] = np.zeros(4, np.float32)
    # attention projections and the second norm gain (act dtype)
    L["Wq"] = to_act(normal(seed, "Wq", (H * dh, d), 0.02), act)
    L["Wk"] = to_act(normal(seed, "Wk", (Hkv * dh, d), 0.02), act)
    L["Wv"] = to_act(normal(seed, "Wv", (Hkv * dh, d), 0.02), act)
    L["Wo"] = to_act(normal(seed, "Wo", (d, H * dh), 0.02), act)
    L["g2"] = to_act(1.0 + normal(seed, "g2", (d,), 0.02), act)
    if with_moe:
        L["Wg"], L["Wu"], L["Wd"] = moe_weights(cfg)
    return L


def dense_variant(L: dict) -> dict:
    """The dense special case of a routed layer (the standard pre-norm
    block): every head in full mode, every token 16-bit, one SwiGLU expert
    (the first), k = 1, the null never chosen, forced through the router
    biases; same shapes and weights otherwise.  Decode workloads' contexts
    become all 16-bit."""
    D = dict(L)
    cfg = dict(L["cfg"], E=1, k=1, experts="dense")
    if "ctx_bits" in cfg:
        cfg["ctx_bits"] = (0.0, 0.0, 0.0, 1.0)
    D["cfg"] = cfg
    H = cfg["H"]
    D["ca"] = np.tile(np.array([-50.0, -50.0, 50.0], np.float32), H)
    D["cb"] = np.array([-50.0, -50.0, -50.0, 50.0], np.float32)
    D["We"] = np.ascontiguousarray(L["We"][:2])
    D["ce"] = np.array([-1.0e4, 50.0], np.float32)
    for n in ("Wg", "Wu", "Wd"):
        D[n] = L[n][:1]
    return D


def granularity_variant(L: dict, groups: int) -> dict:
    """The layer with ``groups`` attention decisions per token instead of one
    per head (groups = 1: a single per-token decision; groups = H_kv: one
    per kv-head group): group a keeps the attention-head rows and biases of
    its first head a H / groups, so its decision is the one that head made
    in the per-head layer.  Same weights and inputs otherwise."""
    cfg = dict(L["cfg"])
    H = cfg["H"]
    assert H % groups == 0
    D = dict(L)
    D["cfg"] = dict(cfg, attn_groups=groups)
    first = np.arange(groups) * (H // groups)
    rows = (3 * first[:, None] + np.arange(3)[None, :]).reshape(-1)
    D["Wa"] = np.ascontiguousarray(L["Wa"][rows])
    D["ca"] = np.ascontiguousarray(L["ca"][rows])
    return D


def make_stack(name: str, n_layers: int, seed: int | None = None) -> list:
    """n_layers routed layers of workload ``name`` for a decode stack: layer 0
    is ``make_layer(name, seed)`` (its x and psi are the stack's inputs);
    layer l > 0 draws its weights and its cached context from the seed
    seed + 7919 l and takes layer 0's calibrated router biases."""
    L0 = make_layer(name, seed)
    out = [L0]
    for l in range(1, n_layers):
        Ll = make_layer(name, L0["cfg"]["seed"] + 7919 * l, biases={})
        for b in ("ca", "ce", "cb"):
            Ll[b] = L0[b].copy()
        out.append(Ll)
    return out


def gumbel(seed, name, shape, *index):
    """Gumbel(0, 1) draws (numpy's inverse-CDF sampler), rounded to fp32."""
    return stream(seed, name, *index).gumbel(0.0, 1.0, shape).astype(np.float32)


def token_positions(cfg: dict) -> np.ndarray:
    """0-based position of every token of a workload: t within its sequence
    (prefill), the context length (decode)."""
    if cfg["kind"] == "prefill":
        return np.tile(np.arange(cfg["T"], dtype=np.int32), cfg["B"]) + np.int32(
            cfg.get("ctx", 0))
    return np.full(cfg["B"], cfg["ctx"], np.int32)


def relax_inputs(L: dict, *, tau_a: float = 1.3, tau_b: float = 0.8,
                 white: bool = True) -> dict:
    """Inputs of the training-time relaxed controller forward of layer ``L``:
    i.i.d. Gumbel(0, 1) noise per attention decision group (3 options) and
    per token for the bit head (4 options); per-axis running whitening
    statistics (mean ~ N(0, 0.1^2), standard deviation ~ U(0.7, 1.3); axis
    order attention, experts, bits); mid-anneal temperatures (the paper
    anneals from 2.0 to 0.5); loss weights, cost targets and dual state."""
    cfg = L["cfg"]
    seed, N = cfg["seed"], len(L["x"])
    A = cfg.get("attn_groups") or cfg["H"]
    R = dict(g_attn=gumbel(seed, "g_attn", (N, A, 3)), g_bits=gumbel(seed, "g_bits", (N, 4)),
             white_mu=None, white_sd=None, white_eps=1e-5, tau_a=tau_a, tau_b=tau_b,
             pos=token_positions(cfg), zeta=0.5, alpha=1e-2, beta=1e-3, gamma=0.1,
             c_target=(0.5, 0.4), dual=(0.3, 0.7, 0.55, 0.45), dual_lr=0.05, dual_ema=0.1)
    if white:
        R["white_mu"] = normal(seed, "white_mu", (3, D_ROUTER), 0.1)
        R["white_sd"] = (np.float32(0.7) + np.float32(0.6) * stream(seed, "white_sd").random(
            (3, D_ROUTER), dtype=np.float32)).astype(np.float32)
    return R


def resample_gumbel_row(seed: int, name: str, token: int, attempt: int, shape) -> np.ndarray:
    """Fresh Gumbel noise for one token's decisions (used to move a relaxed
    decision off a tie)."""
    return stream(seed, name + "_resample", token, attempt).gumbel(0.0, 1.0, shape).astype(
        np.float32)


def moe_weights(cfg: dict):
    """SwiGLU expert weights: gate/up [E, d_ff, d], down [E, d, d_ff]."""
    E, d, dff, seed, act = cfg["E"], cfg["d"], cfg["d_ff"], cfg["seed"], cfg["act"]
    dt = np.float64 if act == "f64" else np.float32
    Wg = np.empty((E, dff, d), dt)
    Wu = np.empty((E, dff, d), dt)
    Wd = np.empty((E, d, dff), dt)
    for e in range(E):
        Wg[e] = to_act(normal(seed, "Wg", (dff, d), 0.02, e), act)
        Wu[e] = to_act(normal(seed, "Wu", (dff, d), 0.02, e), act)
        Wd[e] = to_act(normal(seed, "Wd", (d, dff), 0.02, e), act)
    return Wg, Wu, Wd


def context_bits(cfg: dict, s: int) -> np.ndarray:
    """Exact-count, randomly interleaved bit indices (0..3) of one sequence's
    pre-existing context (decode workloads)."""
    ctx = cfg["ctx"]
    frac = np.asarray(cfg["ctx_bits"], np.float64)
    counts = np.floor(frac * ctx).astype(np.int64)
    rem = ctx - counts.sum()
    order = np.argsort(-(frac * ctx - counts), kind="stable")
    for i in range(rem):
        counts[order[i % 4]] += 1
    bits = np.repeat(np.arange(4, dtype=np.uint8), counts)
    return stream(cfg["seed"], "ctx_bits", s).permutation(bits)


def context_kv(cfg: dict, s: int):
    """Keys (already rotated) and values held in the cache of sequence ``s``
    before the decode step: [ctx, Hkv, dh], N(0, (0.02 sqrt(d))^2), the
    statistics of N(0, 1) states projected by N(0, 0.02^2) weights."""
    ctx, Hkv, dh, d = cfg["ctx"], cfg["Hkv"], cfg["dh"], cfg["d"]
    std = 0.02 * np.sqrt(d)
    k = to_act(normal(cfg["seed"], "ctx_k", (ctx, Hkv, dh), std, s), cfg["act"])
    v = to_act(normal(cfg["seed"], "ctx_v", (ctx, Hkv, dh), std, s), cfg["act"])
    return k, v


def kv_block(seed: int, n: int, Hkv: int, dh: int, act: str, std: float = 1.0,
             tag: str = "kvblock"):
    """Stand-alone K/V tensors [n, Hkv, dh] for appending tests."""
    k = to_act(normal(seed, tag + "_k", (n, Hkv, dh), std), act)
    v = to_act(normal(seed, tag + "_v", (n, Hkv, dh), std), act)
    return k, v
