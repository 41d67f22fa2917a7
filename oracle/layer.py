"""fp64 reference of one TriRoute-routed transformer layer (inference forward).

TEST INFRASTRUCTURE (part of the CPU oracle): only tests, the smoke check and
the benchmark's CPU-baseline leg use it.  It shares no code with the GPU path.

Paper anchors (section / equation names of the TriRoute paper):
  * Sec. 3.1 pre-norm block:  x~ = x + Attn(Norm(x<=t)),  x' = x~ + FFN(Norm(x~)).
  * Sec. 3.2 (A) attention-resolution axis, per head: skip -> 0,
    local -> Attn over a window of w keys, full -> causal attention.
  * Sec. 3.2 (B) expert axis: E experts plus a null expert f_0 = 0; softmax gate
    over {0..E}, top-k set S, weights renormalised over S (null included).
  * Sec. 3.2 (C) KV bit-width axis (see ``quant.py``).
  * Sec. 3.3 controller equation: h = trunk([Norm(x); psi]), h^ = RMSNorm(h),
    z^a = W_a h^, z^e = W_e h^, z^b = W_b h^; trunk = two-layer GELU MLP of
    width 128 (Table 6).
  * Sec. 3.8: inference takes hard argmax decisions and runs only the
    selected computation.
  * Sec. 4 "Models": RoPE, SwiGLU experts, RMSNorm, GQA with H_kv = H/4.

Readings where the paper is silent (each listed in the design notes):
  local window = the w most recent keys [t-w+1, t]; first maximum wins an
  argmax tie; top-k ties go to the lower expert id and the k slots are stored
  in ascending expert id; the null's gate share is dropped, not redistributed;
  RMSNorm eps = 1e-6 with one shared first norm for router and attention;
  exact-erf GELU; rotate-half RoPE with theta = 10000 on the cached (rotated)
  keys; every attention read, including a token's own key, goes through the
  quantized cache (append, then attend).

Precision: the paper's models run in bf16 (Sec. 4 Training).  Read as the
usual mixed-precision contract, every activation tensor handed from one
operator to the next is held in the activation dtype (n1 into the
projections, q/k/v, o, x~, n2 and the SwiGLU product H), while each operator
accumulates in higher precision (here fp64).  ``act = "f64"`` keeps
everything in fp64 (used by the library-reduction pins).
"""
from __future__ import annotations

import numpy as np
import torch
from scipy.special import erf

from . import quant

MODE_SKIP, MODE_LOCAL, MODE_FULL = 0, 1, 2
BITS = quant.BITS
EPS = 1e-6
ROPE_THETA = 10000.0


# ---------------------------------------------------------------- elementwise
def rmsnorm(x, g, eps=EPS):
    """RMSNorm over the last axis (pre-norm of Sec. 3.1; controller h^)."""
    x = np.asarray(x, np.float64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * r * np.asarray(g, np.float64)


def gelu(y):
    """Exact GELU, 0.5 y (1 + erf(y / sqrt 2)) (trunk activation, Table 6)."""
    y = np.asarray(y, np.float64)
    return 0.5 * y * (1.0 + erf(y / np.sqrt(2.0)))


def silu(u):
    """SiLU, u / (1 + exp(-u)), the SwiGLU expert gate (Sec. 4 Models)."""
    u = np.asarray(u, np.float64)
    return u / (1.0 + np.exp(-u))


def softmax(z, axis=-1):
    z = np.asarray(z, np.float64)
    m = np.max(z, axis=axis, keepdims=True)
    e = np.exp(z - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def rope(x, pos, theta=ROPE_THETA):
    """Rotate-half RoPE.  ``x`` [..., n, heads, dh], ``pos`` [n]:
    pair (j, j + dh/2) is rotated by angle pos * theta^(-2j/dh)."""
    x = np.asarray(x, np.float64)
    dh = x.shape[-1]
    half = dh // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / dh)
    ang = np.asarray(pos, np.float64)[:, None] * inv[None, :]       # [n, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


def to_native(a, act):
    """Round to the activation dtype: the precision of every tensor handed
    between operators, and the "native precision" of a 16-bit cache entry."""
    t = torch.from_numpy(np.ascontiguousarray(a, np.float64))
    if act == "bf16":
        return t.to(torch.bfloat16).to(torch.float32).numpy()
    if act == "f32":
        return t.to(torch.float32).numpy()
    return t.numpy()


# -------------------------------------------------------------- controller
def router_logits(L, tokens=None):
    """Controller equation (Sec. 3.3) on tokens ``tokens`` (all by default).

    Returns n1 (the shared first norm), z^a [n, A, 3], z^e [n, E+1], z^b [n, 4]
    with A attention decisions per token (``cfg["attn_groups"]``, default H:
    one per head; Sec. 3.2 (A) routes per head or per head group).
    Whitening and the gradient-balance scale are frozen at inference and are
    already folded into (W, c).
    """
    cfg = L["cfg"]
    x = L["x"] if tokens is None else L["x"][tokens]
    psi = L["psi"] if tokens is None else L["psi"][tokens]
    n1 = rmsnorm(x, L["g1"])
    s = np.concatenate([n1, np.asarray(psi, np.float64)], axis=1)
    u = gelu(s @ np.asarray(L["W1"], np.float64).T + L["b1"])
    h = u @ np.asarray(L["W2"], np.float64).T + L["b2"]
    hh = rmsnorm(h, L["gr"])
    za = (hh @ np.asarray(L["Wa"], np.float64).T + L["ca"]).reshape(
        len(x), cfg.get("attn_groups") or cfg["H"], 3)
    ze = hh @ np.asarray(L["We"], np.float64).T + L["ce"]
    zb = hh @ np.asarray(L["Wb"], np.float64).T + L["cb"]
    return n1, za, ze, zb


def _argmax_first(row):
    best = 0
    for j in range(1, len(row)):
        if row[j] > row[best]:
            best = j
    return best


def decide(za, ze, zb, k, H=None):
    """Hard inference decisions (Sec. 3.8, Sec. 3.2 (A)-(C)).

    mode[i, h] = argmax over (skip, local, full) of the logits of h's
    decision group (za [N, A, 3]: query heads h with h // (H / A) == a share
    group a; A = H, the default, is one decision per head); bit[i] = argmax
    over (2, 4, 8, 16) as index 0..3; S_i = the k most probable options of
    softmax(z^e) (index 0 = null), gates p_j / sum_{S_i} p.
    """
    N, A, _ = za.shape
    H = A if H is None else H
    assert H % A == 0
    mode = np.zeros((N, H), np.uint8)
    bit = np.zeros(N, np.uint8)
    eidx = np.zeros((N, k), np.int32)
    egate = np.zeros((N, k), np.float64)
    p = softmax(ze, axis=-1)
    for i in range(N):
        for h in range(H):
            mode[i, h] = _argmax_first(za[i, h // (H // A)])
        bit[i] = _argmax_first(zb[i])
        # larger probability first, lower index on ties
        order = sorted(range(p.shape[1]), key=lambda j: (-p[i, j], j))
        chosen = sorted(order[:k])
        tot = sum(p[i, j] for j in chosen)
        for sl, j in enumerate(chosen):
            eidx[i, sl] = j
            egate[i, sl] = p[i, j] / tot
    return mode, bit, eidx, egate


def margins(za, ze, zb, k):
    """Smallest logit gap that decides each token's routing (argmax gaps per
    head and for bits, and the k-th vs (k+1)-th expert logit gap)."""
    def gap_top1(z):
        s = np.sort(z, axis=-1)
        return s[..., -1] - s[..., -2]
    ga = gap_top1(za).min(axis=1)
    gb = gap_top1(zb)
    se = np.sort(ze, axis=-1)
    ge = se[:, -k] - se[:, -k - 1]
    return np.minimum(np.minimum(ga, gb), ge)


# -------------------------------------------------------------- compaction
def compact(mode, eidx, B, T, H, E, k):
    """Deterministic stable partitions (plain loops).

    Attention: for segment s = (b*H + h)*2 + (m-1), m in {local, full}, the
    ascending t with mode[b*T+t, h] == m.  Experts: for e = 1..E the ascending
    assignment ids a = i*k + slot with eidx[i, slot] == e.  ``exp_cnt[0]``
    counts null assignments (they are never listed).
    """
    nseg = B * H * 2
    attn_cnt = np.zeros(nseg, np.int32)
    attn_idx = np.full((nseg, T), -1, np.int32)
    for b in range(B):
        for h in range(H):
            for t in range(T):
                m = int(mode[b * T + t, h])
                if m == MODE_SKIP:
                    continue
                s = (b * H + h) * 2 + (m - 1)
                attn_idx[s, attn_cnt[s]] = t
                attn_cnt[s] += 1
    N = B * T
    exp_cnt = np.zeros(E + 1, np.int32)
    lists = [[] for _ in range(E + 1)]
    for i in range(N):
        for sl in range(k):
            e = int(eidx[i, sl])
            exp_cnt[e] += 1
            lists[e].append(i * k + sl)
    exp_off = np.zeros(E + 1, np.int32)
    for e in range(1, E + 1):
        exp_off[e] = exp_off[e - 1] + exp_cnt[e]
    exp_rows = np.array([a for e in range(1, E + 1) for a in lists[e]], np.int32)
    return dict(attn_cnt=attn_cnt, attn_idx=attn_idx, exp_cnt=exp_cnt,
                exp_off=exp_off, exp_rows=exp_rows)


# ------------------------------------------------------------ attention
def qkv(n1, L, pos, act=None):
    """q = Wq n1, k = Wk n1, v = Wv n1 per head, RoPE on q and k at ``pos``;
    outputs held in the activation dtype (``act``, default the workload's)."""
    cfg = L["cfg"]
    H, Hkv, dh = cfg["H"], cfg["Hkv"], cfg["dh"]
    act = act or cfg["act"]
    n = len(n1)
    q = (n1 @ np.asarray(L["Wq"], np.float64).T).reshape(n, H, dh)
    k = (n1 @ np.asarray(L["Wk"], np.float64).T).reshape(n, Hkv, dh)
    v = (n1 @ np.asarray(L["Wv"], np.float64).T).reshape(n, Hkv, dh)
    return (to_native(rope(q, pos), act), to_native(rope(k, pos), act),
            to_native(v, act))


def store_kv(k, v, bit, cfg):
    """Write tokens into the cache at their chosen width (Sec. 3.2 (C)).

    ``k``/``v`` [n, Hkv, dh] are the native-precision values.  Returns the
    read-back values k^, v^ (fp64) and, per width, the codes and fp16
    scale/zero of the tokens stored at that width.
    """
    G = cfg["G"]
    khat = np.zeros(k.shape, np.float64)
    vhat = np.zeros(v.shape, np.float64)
    stored = {}
    for bi, b in enumerate(BITS):
        sel = np.flatnonzero(bit == bi)
        if len(sel) == 0:
            continue
        kc, ks, kz = quant.quantize(k[sel], b, G)
        vc, vs, vz = quant.quantize(v[sel], b, G)
        if b == 16:
            khat[sel] = k[sel]
            vhat[sel] = v[sel]
        else:
            khat[sel] = quant.dequantize(kc, ks, kz, G)
            vhat[sel] = quant.dequantize(vc, vs, vz, G)
        stored[bi] = dict(tokens=sel, kc=kc, ks=ks, kz=kz, vc=vc, vs=vs, vz=vz)
    return khat, vhat, stored


def attention_seq(q, qpos, khat, vhat, modes, w):
    """Routed attention of one sequence (Sec. 3.2 (A)).

    ``q`` [nq, H, dh] at positions ``qpos``; keys/values [P, Hkv, dh] of the
    same sequence at positions 0..P-1 (already read back from the cache);
    ``modes`` [nq, H].  Query head h reads kv head floor(h / (H / Hkv)).
    skip -> 0; local -> keys [t-w+1, t]; full -> keys [0, t].
    """
    nq, H, dh = q.shape
    P, Hkv, _ = khat.shape
    grp = H // Hkv
    out = np.zeros((nq, H, dh), np.float64)
    j = np.arange(P)[None, :]
    t = np.asarray(qpos)[:, None]
    for h in range(H):
        g = h // grp
        m = modes[:, h][:, None]
        lo = np.where(m == MODE_LOCAL, np.maximum(t - w + 1, 0), 0)
        allowed = (j <= t) & (j >= lo) & (m != MODE_SKIP)
        sc = (q[:, h, :] @ khat[:, g, :].T) / np.sqrt(dh)
        sc = np.where(allowed, sc, -np.inf)
        rows = allowed.any(axis=1)
        if not rows.any():
            continue
        p = softmax(sc[rows], axis=-1)
        out[rows, h, :] = p @ vhat[:, g, :]
    return out


def oproj(x, o, Wo):
    """x~ = x + W_o concat_h(o_h) (first residual of Sec. 3.1)."""
    n = len(x)
    return np.asarray(x, np.float64) + o.reshape(n, -1) @ np.asarray(Wo, np.float64).T


def moe(xt, L, eidx, egate, act=None):
    """Second half of the block: x' = x~ + sum_{j in S, j != 0} g_j f_j(Norm x~)
    with SwiGLU experts f_j(u) = W_down,j (silu(W_gate,j u) * W_up,j u).
    The null expert contributes nothing (Sec. 3.2 (B)).  n2 and the SwiGLU
    product are held in ``act`` (default the workload's activation dtype)."""
    cfg = L["cfg"]
    act = act or cfg["act"]
    n2 = to_native(rmsnorm(xt, L["g2"]), act)
    y = np.zeros_like(n2)
    k = eidx.shape[1]
    for e in range(1, cfg["E"] + 1):
        hit = np.argwhere(eidx == e)
        if len(hit) == 0:
            continue
        rows, slots = hit[:, 0], hit[:, 1]
        Wg = np.asarray(L["Wg"][e - 1], np.float64)
        Wu = np.asarray(L["Wu"][e - 1], np.float64)
        Wd = np.asarray(L["Wd"][e - 1], np.float64)
        u = n2[rows]
        hmid = to_native(silu(u @ Wg.T) * (u @ Wu.T), act)
        np.add.at(y, rows, egate[rows, slots][:, None] * (hmid @ Wd.T))
    del k
    return xt + y, n2, y


# ------------------------------------------------------------ whole layer
def layer_prefill(L, rows=None, kv_in=None, xt_in=None, o_in=None, round_act=True):
    """Prefill of B fresh sequences of T tokens (cache empty beforehand).

    ``rows``: token indices whose attention / FFN outputs are wanted (all by
    default).  Routing and compaction are always computed for every token;
    K/V are computed and stored for every token of the sequences ``rows``
    touch.

    Discretely forced evaluation (the comparison protocol for results that a
    legitimate one-ulp difference upstream can move):
      * ``kv_in``: {b: (k, v)} native-precision [T, Hkv, dh] keys (rotated) and
        values of sequence b to quantize into the cache in place of the
        oracle's own projections; the oracle's quantizer and dequantizer
        still do all of the cache arithmetic;
      * ``o_in``: [len(rows), H * dh] attention outputs to feed the output
        projection in place of the oracle's own o (the returned ``o`` stays the
        oracle's);
      * ``xt_in``: [len(rows), d] first-residual outputs to feed the expert
        block in place of the oracle's own x~.
    ``round_act=False`` holds every tensor handed between operators in fp64
    instead of the activation dtype (the quantizer still works in fp32).
    """
    cfg = L["cfg"]
    B, T, H, w = cfg["B"], cfg["T"], cfg["H"], cfg["w"]
    act = cfg["act"] if round_act else "f64"
    N = B * T
    n1, za, ze, zb = router_logits(L)
    mode, bit, eidx, egate = decide(za, ze, zb, cfg["k"], cfg["H"])
    cmp = compact(mode, eidx, B, T, H, cfg["E"], cfg["k"])
    rows = np.arange(N) if rows is None else np.asarray(sorted(set(rows)))
    seqs = sorted(set(int(r) // T for r in rows))
    q_all, k_all, v_all, o_rows = {}, {}, {}, {}
    stored = {}
    n1a = to_native(n1, act)
    for b in seqs:
        sl = slice(b * T, (b + 1) * T)
        pos = np.arange(T)
        q, kn, vn = qkv(n1a[sl], L, pos, act)
        kst, vst = (kn, vn) if kv_in is None else kv_in[b]
        khat, vhat, st = store_kv(kst, vst, bit[sl], cfg)
        stored[b] = st
        want = [int(r) - b * T for r in rows if int(r) // T == b]
        o = attention_seq(q[want], np.asarray(want), khat, vhat,
                          mode[sl][want], w)
        for ti, t in enumerate(want):
            o_rows[b * T + t] = o[ti]
        q_all[b], k_all[b], v_all[b] = q, kn, vn
    o = to_native(np.stack([o_rows[int(r)] for r in rows]), act)
    oin = o if o_in is None else np.asarray(o_in, np.float64)
    xt = to_native(oproj(L["x"][rows], oin, L["Wo"]), act)
    xin = xt if xt_in is None else np.asarray(xt_in, np.float64)
    xout, n2, y = moe(xin, L, eidx[rows], egate[rows], act)
    return dict(rows=rows, n1=n1, za=za, ze=ze, zb=zb, mode=mode, bit=bit,
                eidx=eidx, egate=egate, cmp=cmp, q=q_all, k=k_all, v=v_all,
                stored=stored, o=o, xt=xt, n2=n2, y=y, xout=xout)


def decode_cache_seq(cfg, s, context=None):
    """Read-back values of sequence ``s``'s pre-existing context (decode
    workloads): native-precision K/V [ctx, Hkv, dh] and per-position widths
    from ``context(s) -> (k, v, bits)`` (default: the generator's context),
    stored through the quantizer."""
    if context is None:
        import gen
        k, v = gen.context_kv(cfg, s)
        bits = gen.context_bits(cfg, s)
    else:
        k, v, bits = context(s)
    khat, vhat, stored = store_kv(k, v, bits, cfg)
    return khat, vhat, stored, bits


def layer_decode(L, seqs=None, context=None, kv_in=None, xt_in=None, o_in=None,
                 round_act=True):
    """One decode step: each sequence b gets one new token at position
    P = ctx; its K/V are appended at the routed width, then its query heads
    attend over the read-back cache [0, P] (or its last w keys).

    ``context``: as in ``decode_cache_seq``.  ``kv_in`` ({s: (k, v)}, each
    [1, Hkv, dh]), ``o_in``, ``xt_in`` and ``round_act``: as in
    ``layer_prefill``."""
    cfg = L["cfg"]
    B, H, w, ctx = cfg["B"], cfg["H"], cfg["w"], cfg["ctx"]
    act = cfg["act"] if round_act else "f64"
    n1, za, ze, zb = router_logits(L)
    mode, bit, eidx, egate = decide(za, ze, zb, cfg["k"], cfg["H"])
    cmp = compact(mode, eidx, B, 1, H, cfg["E"], cfg["k"])
    seqs = list(range(B)) if seqs is None else sorted(set(int(s) for s in seqs))
    rows = np.asarray(seqs)
    pos = np.full(len(rows), ctx)
    q, kn, vn = qkv(to_native(n1[rows], act), L, pos, act)
    o = np.zeros((len(rows), H, cfg["dh"]))
    new_stored = {}
    for ri, s in enumerate(seqs):
        khat, vhat, _, _ = decode_cache_seq(cfg, s, context)
        kst, vst = (kn[ri:ri + 1], vn[ri:ri + 1]) if kv_in is None else kv_in[s]
        kh1, vh1, st = store_kv(kst, vst, bit[s:s + 1], cfg)
        new_stored[s] = st
        khat = np.concatenate([khat, kh1], axis=0)
        vhat = np.concatenate([vhat, vh1], axis=0)
        o[ri] = attention_seq(q[ri:ri + 1], np.array([ctx]), khat, vhat,
                              mode[s:s + 1], w)[0]
        del khat, vhat
    o = to_native(o, act)
    oin = o if o_in is None else np.asarray(o_in, np.float64)
    xt = to_native(oproj(L["x"][rows], oin, L["Wo"]), act)
    xin = xt if xt_in is None else np.asarray(xt_in, np.float64)
    xout, n2, y = moe(xin, L, eidx[rows], egate[rows], act)
    return dict(rows=rows, n1=n1, za=za, ze=ze, zb=zb, mode=mode, bit=bit,
                eidx=eidx, egate=egate, cmp=cmp, q=q, k=kn, v=vn,
                stored=new_stored, o=o, xt=xt, n2=n2, y=y, xout=xout)
