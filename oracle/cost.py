"""Hard-decision cost accounting of one routed layer.

TEST INFRASTRUCTURE (part of the CPU oracle): only tests use it.  It shares
no code with the GPU path.

Paper anchors:
  * Sec. 3.5 cost model, per token t and layer: attention read
    kappa^a(t) = 0 (skip), ~2 d min(t, w) (local), ~2 d t (full), counted in
    key interactions; active experts kappa^e ~ 3 d d_f per SwiGLU expert;
    KV memory 2 d_kv b bits for a token stored at width b.
  * Sec. 3.8 / App. A: at inference the hard argmax decisions replace the
    soft expectations, so the accounted cost is the executed one; App. A's
    dense reference is full attention, the full FFN and a 16-bit cache,
    sum_t (2 d t + 3 d d_f) FLOP-units and sum_t 2 d_kv 16 bits.

Decisions are per (token, head) for attention (the per-head mode axis of
Sec. 3.2 (A)), so a head contributes 2 d_h per key it reads and the sum over
the H heads of a token in one mode is the paper's 2 d per key.  t counts the
keys a full query reads: the query at 0-based position P reads P + 1 keys.

Readings (listed in the design notes): R1, a local query reads the w most
recent keys [P - w + 1, P], so min(P + 1, w) of them; R27, executed expert
cost counts each real expert of S_t once (the null expert is never
materialized, Sec. 3.8), without the relaxed cost's gate weights.
"""
import numpy as np

from .layer import BITS, MODE_FULL, MODE_LOCAL, MODE_SKIP


def key_interactions(mode, qpos, w):
    """[N, H] number of keys each (token, head) reads: 0 (skip), min(P + 1, w)
    (local), P + 1 (full), P = qpos[token]."""
    mode = np.asarray(mode)
    t = np.asarray(qpos, np.int64)[:, None] + 1
    return np.where(mode == MODE_FULL, t,
                    np.where(mode == MODE_LOCAL, np.minimum(t, w), 0)).astype(np.int64)


def cost_terms(cfg, mode, bit, eidx, qpos):
    """Accounted cost of N tokens' hard decisions (Sec. 3.5, hard form):

    keys       total key interactions (sum over tokens and heads);
    attn       sum over (token, head) of 2 d_h keys (multiply-accumulates);
    kv_bits    sum over tokens of 2 d_kv b_t (the cache codes the tokens add);
    experts    number of real expert assignments (R27);
    ffn        3 d d_f per real assignment.
    ``bit``: width indices 0..3 (2, 4, 8, 16 bits); ``eidx`` [N, k] expert ids
    (0 = null)."""
    dh, d, dff = cfg["dh"], cfg["d"], cfg["d_ff"]
    dkv = cfg["Hkv"] * dh
    keys = key_interactions(mode, qpos, cfg["w"])
    widths = np.asarray(BITS, np.int64)[np.asarray(bit, np.int64)]
    experts = int((np.asarray(eidx) != 0).sum())
    return dict(keys=int(keys.sum()), attn=2 * dh * int(keys.sum()),
                kv_bits=int(2 * dkv * widths.sum()), experts=experts,
                ffn=3 * d * dff * experts)


def dense_reference(cfg, qpos):
    """App. A dense reference of the same tokens: full attention in every
    head, one full FFN per token, a 16-bit cache."""
    qpos = np.asarray(qpos, np.int64)
    H, dh, d, dff = cfg["H"], cfg["dh"], cfg["d"], cfg["d_ff"]
    keys = H * int((qpos + 1).sum())
    return dict(keys=keys, attn=2 * dh * keys, kv_bits=int(2 * cfg["Hkv"] * dh * 16 * len(qpos)),
                experts=len(qpos), ffn=3 * d * dff * len(qpos))


__all__ = ["key_interactions", "cost_terms", "dense_reference", "MODE_SKIP"]
