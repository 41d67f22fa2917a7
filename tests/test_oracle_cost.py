"""Pins of the oracle's hard-decision cost accounting (Sec. 3.5 cost model,
App. A dense reference) against brute force and closed forms."""
import numpy as np
import pytest

import gen
import oracle
from oracle import cost


def _brute_keys(mode, qpos, w):
    """Keys each (token, head) may read, by testing every cached position."""
    N, H = mode.shape
    out = np.zeros((N, H), np.int64)
    for n in range(N):
        P = int(qpos[n])
        for h in range(H):
            for j in range(P + 1):
                m = mode[n, h]
                if m == oracle.MODE_FULL or (m == oracle.MODE_LOCAL and j >= P - w + 1):
                    out[n, h] += 1
    return out


def test_key_interactions_brute_force():
    rng = np.random.default_rng(3)
    for w in (1, 4, 7, 64):
        mode = rng.integers(0, 3, (90, 5))
        qpos = np.sort(rng.choice(200, 90, replace=False))
        np.testing.assert_array_equal(cost.key_interactions(mode, qpos, w),
                                      _brute_keys(mode, qpos, w))


@pytest.mark.parametrize("T,w,H", [(1, 3, 2), (50, 7, 3), (300, 128, 4)])
def test_closed_forms(T, w, H):
    cfg = dict(H=H, Hkv=1, dh=64, d=64 * H, d_ff=128, w=w)
    qpos = np.arange(T)
    full = cost.cost_terms(cfg, np.full((T, H), 2), np.full(T, 3), np.ones((T, 1)), qpos)
    assert full["keys"] == H * T * (T + 1) // 2
    loc = cost.cost_terms(cfg, np.full((T, H), 1), np.zeros(T, int), np.zeros((T, 2)), qpos)
    m = min(T, w)
    assert loc["keys"] == H * (m * (m + 1) // 2 + (T - m) * w)
    assert loc["kv_bits"] == T * 2 * 64 * 2 and loc["experts"] == 0 and loc["ffn"] == 0
    skip = cost.cost_terms(cfg, np.zeros((T, H)), np.full(T, 1), np.zeros((T, 2)), qpos)
    assert skip["keys"] == 0 and skip["kv_bits"] == T * 2 * 64 * 4
    # the dense special case is App. A's dense reference, term for term
    assert full == cost.dense_reference(cfg, qpos)


def test_mixed_decisions_sum_per_token():
    rng = np.random.default_rng(5)
    cfg = dict(H=4, Hkv=2, dh=32, d=128, d_ff=256, w=16)
    N = 77
    mode, bit = rng.integers(0, 3, (N, 4)), rng.integers(0, 4, N)
    eidx = rng.integers(0, 5, (N, 2))
    eidx[3] = 0  # a token whose two slots are both null costs no expert (R27)
    qpos = 1000 + np.arange(N)
    c = cost.cost_terms(cfg, mode, bit, eidx, qpos)
    kv = sum(2 * 2 * 32 * (2, 4, 8, 16)[b] for b in bit)
    ex = sum(int(e != 0) for row in eidx for e in row)
    assert c["kv_bits"] == kv and c["experts"] == ex and c["ffn"] == 3 * 128 * 256 * ex
    assert c["attn"] == 2 * 32 * int(_brute_keys(mode, qpos, 16).sum())


def test_dense_variant_decisions_cost_the_dense_reference():
    """The generator's dense variant of a workload decides full / 16-bit /
    one expert for every token, so its accounted cost is App. A's reference."""
    L = gen.dense_variant(gen.make_layer("tiny_f32_prefill", act="f64"))
    n1, za, ze, zb = oracle.router_logits(L)
    mode, bit, eidx, egate = oracle.decide(za, ze, zb, L["cfg"]["k"], L["cfg"]["H"])
    qpos = np.arange(L["cfg"]["T"])
    assert cost.cost_terms(L["cfg"], mode, bit, eidx, qpos) == cost.dense_reference(L["cfg"], qpos)
