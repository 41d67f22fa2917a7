"""Executed work of the GPU layer against the accounted cost.

Sec. 3.8 and App. A: at inference the hard decisions replace the soft
expectations of the Sec. 3.5 cost model, and only the selected computation
runs, so the accounted cost equals the executed one.  Here "accounted" is the
oracle's cost of its own decisions (oracle.cost, pinned on the CPU) and
"executed" is read off the GPU after the layer call:

* key interactions: for every (token, head) of the GPU's mode taps, the
  cached keys of the token's sequence whose positions the attention reads
  (skip: none; local: [P - w + 1, P]; full: [0, P]), counted in the GPU
  cache's own position arrays after the call.  That the attention reads
  exactly those keys is what the attention parity tests establish;
* KV memory: the GPU cache's pool lengths times 2 d_kv b bits (codes; the
  fp16 scale/zero words are reported beside them);
* experts: the real (non-null) expert slots of the GPU's routing taps.

Integers, compared exactly; routed/dense ratios against App. A's dense
reference are recorded."""
import numpy as np
import pytest
import torch

import gen
import oracle
import paper_2607_06601_amd as tr
from oracle import cost
from paper_2607_06601_amd.device import DeviceLayer

from _common import layer, note, npy
from test_gpu_layer import _taps, export_pool, fill_context

pytestmark = pytest.mark.gpu
DEV = "cuda"
BITS = np.array([2, 4, 8, 16])


def _cached_positions(c, cache, cfg, s):
    """Sorted positions of every key cached for sequence s, and the pool lengths."""
    pl = npy(cache.pool_len())[s].astype(np.int64)
    pos = [export_pool(c, cache, s, bi, int(pl[bi]), cfg["act"], cfg["Hkv"], cfg["dh"], cfg["G"])[4]
           for bi in range(4) if pl[bi] > 0]
    return np.sort(np.concatenate(pos)), pl


def _executed_keys(mode, qpos, positions, w):
    """Cached keys read by each (token, head) of one sequence."""
    P = np.asarray(qpos, np.int64)[:, None]
    lo = np.where(mode == oracle.MODE_LOCAL, P - w + 1, 0)
    n = np.searchsorted(positions, P, side="right") - np.searchsorted(positions, lo, side="left")
    return np.where(mode == oracle.MODE_SKIP, 0, n)


def _check(cfg, name, mode_g, eidx_g, caches, qpos_of, acc, dense):
    """caches: {s: (positions, pool lengths)}; qpos_of(s) -> (rows, positions)."""
    keys = kv_bits = meta_bits = 0
    dkv = cfg["Hkv"] * cfg["dh"]
    ng = cfg["dh"] // cfg["G"]
    for s, (positions, pl) in caches.items():
        rows, qpos = qpos_of(s)
        keys += int(_executed_keys(mode_g[rows], qpos, positions, cfg["w"]).sum())
        kv_bits += int((pl * 2 * dkv * BITS).sum())
        meta_bits += int(pl[:3].sum()) * 2 * cfg["Hkv"] * ng * 2 * 16
    experts = int((eidx_g != 0).sum())
    assert keys == acc["keys"], (keys, acc["keys"])
    assert kv_bits == acc["kv_bits"], (kv_bits, acc["kv_bits"])
    assert experts == acc["experts"], (experts, acc["experts"])
    note(f"{name}: executed = accounted: keys {keys}, KV code bits {kv_bits} (+ scale/zero "
         f"{meta_bits}), expert slots {experts}", 0.0)
    for k in ("attn", "kv_bits", "ffn"):
        note(f"{name}: routed / dense {k}", acc[k] / dense[k])


@pytest.mark.parametrize("name,seed", [("160m_bf16_prefill", 1), ("1p3b_bf16_prefill", 104)])
def test_prefill_executed_equals_accounted(name, seed):
    L = layer(name, seed)
    cfg = L["cfg"]
    B, T = cfg["B"], cfg["T"]
    D = DeviceLayer(L)
    c = D.cfg
    cache = tr.KVCache(c, B, T)
    t, s = _taps(cfg, B * T, D.act)
    xo = torch.empty(B * T, cfg["d"], dtype=D.act, device=DEV)
    tr.layer_prefill(c, B, T, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo,
                     tr.workspace(c, tr.OP_LAYER_PREFILL, B, T), taps=s)
    torch.cuda.synchronize()
    _, za, ze, zb = oracle.router_logits(L)
    mode, bit, eidx, _ = oracle.decide(za, ze, zb, cfg["k"], cfg["H"])
    qpos = np.tile(np.arange(T), B)
    acc = cost.cost_terms(cfg, mode, bit, eidx, qpos)
    caches = {}
    for b in range(B):
        positions, pl = _cached_positions(c, cache, cfg, b)
        np.testing.assert_array_equal(positions, np.arange(T))  # every token once
        caches[b] = (positions, pl)
    _check(cfg, name, npy(t["mode"]), npy(t["eidx"]), caches,
           lambda b: (np.arange(b * T, (b + 1) * T), np.arange(T)), acc,
           cost.dense_reference(cfg, qpos))


def test_decode_executed_equals_accounted():
    name = "1p3b_bf16_decode"
    L = layer(name)
    cfg = L["cfg"]
    B, ctx = cfg["B"], cfg["ctx"]
    D = DeviceLayer(L)
    c = D.cfg
    cache = tr.KVCache(c, B, ctx + 16)
    fill_context(c, cache, cfg, D.act)
    t, s = _taps(cfg, B, D.act)
    xo = torch.empty(B, cfg["d"], dtype=D.act, device=DEV)
    tr.layer_decode(c, B, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo,
                    tr.workspace(c, tr.OP_LAYER_DECODE, B, 1), taps=s)
    torch.cuda.synchronize()
    _, za, ze, zb = oracle.router_logits(L)
    mode, bit, eidx, _ = oracle.decide(za, ze, zb, cfg["k"], cfg["H"])
    # the step's cost: its new tokens, each reading the context plus itself;
    # the KV term counts the step's own token (the context was stored before)
    qpos = np.full(B, ctx)
    acc = cost.cost_terms(cfg, mode, bit, eidx, qpos)
    ctx_bits = sum(int((2 * cfg["Hkv"] * cfg["dh"] * BITS[gen.context_bits(cfg, b)]).sum())
                   for b in range(B))
    acc = dict(acc, kv_bits=acc["kv_bits"] + ctx_bits)
    caches = {b: _cached_positions(c, cache, cfg, b) for b in range(B)}
    for b in range(B):
        np.testing.assert_array_equal(caches[b][0], np.arange(ctx + 1))
    dense = dict(cost.dense_reference(cfg, qpos),
                 kv_bits=B * (ctx + 1) * 2 * cfg["Hkv"] * cfg["dh"] * 16)
    _check(cfg, name, npy(t["mode"]), npy(t["eidx"]), caches,
           lambda b: (np.array([b]), np.array([ctx])), acc, dense)
