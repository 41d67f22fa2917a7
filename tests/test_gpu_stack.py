"""A decode step through a stack of routed layers on the GPU
(triroute_stack_decode; Sec. 3.3 side features carrying the previous layer's
decisions, Sec. 3.8 per-layer decisions in one pass).

1. The stack equals, bit for bit, the same layers run one triroute_layer_decode
   call at a time, each fed the previous call's output and side features
   built from the previous call's decision taps by the oracle's rule (so the
   device-side feature kernel and the buffers handed between layers are what
   is checked);
2. every layer of that layer-by-layer run against the oracle with the
   protocol of test_layer_decode, forced at the layer's input (the GPU's
   output of the layer before): decisions bit exact on every token whose
   deciding logit gap clears 1e-4 (the inputs of layers past the first are
   not steered away from ties), the new token's cache codes bit exact, and
   o, x~, x_out within tolerance."""
import numpy as np
import pytest
import torch

import gen
import oracle
import paper_2607_06601_amd as tr
from oracle import stack
from oracle.ties import DELTA, enforce_margins
from paper_2607_06601_amd.device import DeviceLayer, to_dev

from _common import assert_close, note, npy
from test_gpu_layer import _taps, check_pool, fill_context

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _caches(Ds, Ls):
    out = []
    for D, L in zip(Ds, Ls):
        cfg = L["cfg"]
        cache = tr.KVCache(D.cfg, cfg["B"], cfg["ctx"] + 16)
        fill_context(D.cfg, cache, cfg, D.act)
        out.append(cache)
    return out


@pytest.mark.parametrize("name,n_layers,nseq", [("410m_bf16_decode", 3, 4)])
def test_stack_decode(name, n_layers, nseq):
    Ls = gen.make_stack(name, n_layers)
    enforce_margins(Ls[0])
    cfg = Ls[0]["cfg"]
    act, B, ctx, Hkv, dh, H, k = (cfg[x] for x in ("act", "B", "ctx", "Hkv", "dh", "H", "k"))
    Ds = [DeviceLayer(L) for L in Ls]
    c = Ds[0].cfg
    # 1: the stack against the layer-by-layer run
    caches = _caches(Ds, Ls)
    xo = torch.empty(B, cfg["d"], dtype=Ds[0].act, device=DEV)
    tr.stack_decode(c, B, Ds[0].x, Ds[0].psi, [(D.rw, D.dw, D.mw) for D in Ds], caches, xo,
                    tr.workspace(c, tr.OP_STACK_DECODE, B, 1))
    torch.cuda.synchronize()
    assert all(ca.status() == 0 for ca in caches)
    del caches
    caches = _caches(Ds, Ls)
    psi0 = np.asarray(Ls[0]["psi"], np.float64)
    x, psi = Ds[0].x, Ds[0].psi
    per = []
    for l, (D, L) in enumerate(zip(Ds, Ls)):
        t, s = _taps(cfg, B, D.act)
        xl = torch.empty(B, cfg["d"], dtype=D.act, device=DEV)
        tr.layer_decode(c, B, x, psi, D.rw, D.dw, D.mw, caches[l], xl,
                        tr.workspace(c, tr.OP_LAYER_DECODE, B, 1), taps=s)
        torch.cuda.synchronize()
        per.append((x, psi, t, xl))
        nxt = stack.psi_next(psi0, npy(t["mode"]), npy(t["bit"]), npy(t["eidx"]))
        x, psi = xl, to_dev(nxt.astype(np.float32), torch.float32)
    assert torch.equal(xo, per[-1][3])
    # 2: each layer against the oracle, forced at its input
    seqs = sorted({0, B - 1} | set(int(v) for v in gen.stream(cfg["seed"], "stack_seqs").choice(
        B, nseq, replace=False)))
    for l, ((xin, pin, t, xl), L, D) in enumerate(zip(per, Ls, Ds)):
        cfg_l = L["cfg"]
        Ll = dict(L, x=npy(xin).astype(np.float64), psi=npy(pin).astype(np.float64))
        _, za, ze, zb = oracle.router_logits(Ll)
        ok = oracle.margins(za, ze, zb, k) >= DELTA
        note(f"layer {l}: tokens within {DELTA} of a routing tie (excluded)", float((~ok).sum()))
        cmp_seqs = [s_ for s_ in seqs if ok[s_]]
        assert len(cmp_seqs) >= 2
        r0 = oracle.layer_decode(Ll, cmp_seqs)
        for key in ("mode", "bit", "eidx"):
            np.testing.assert_array_equal(npy(t[key])[ok], r0[key][ok])
        np.testing.assert_allclose(npy(t["egate"])[ok], r0["egate"][ok], rtol=2e-5, atol=1e-6)
        gq, gk, gv = (npy(t[key])[cmp_seqs] for key in ("q", "k", "v"))
        assert_close(gq, r0["q"].reshape(len(cmp_seqs), -1), act, f"layer {l} q")
        assert_close(gk, r0["k"].reshape(len(cmp_seqs), -1), act, f"layer {l} k")
        assert_close(gv, r0["v"].reshape(len(cmp_seqs), -1), act, f"layer {l} v")
        kv_in = {s_: (gk[i].reshape(1, Hkv, dh), gv[i].reshape(1, Hkv, dh))
                 for i, s_ in enumerate(cmp_seqs)}
        gxt = npy(t["xt"])[cmp_seqs]
        r1 = oracle.layer_decode(Ll, cmp_seqs, kv_in=kv_in, o_in=npy(t["o"])[cmp_seqs], xt_in=gxt)
        bits_new = npy(t["bit"])
        for s_ in cmp_seqs:
            _, _, _, bits = oracle.decode_cache_seq(cfg_l, s_)
            bi = int(bits_new[s_])
            check_pool(c, caches[l], cfg_l, s_, bi, r1["stored"][s_][bi], [ctx],
                       first=int((bits == bi).sum()))
        assert_close(npy(t["o"])[cmp_seqs], r1["o"].reshape(len(cmp_seqs), -1), act,
                     f"layer {l} o (forced codes)")
        assert_close(gxt, r1["xt"], act, f"layer {l} x~ (forced o)")
        assert_close(npy(xl)[cmp_seqs], r1["xout"], act, f"layer {l} x_out (forced x~)")
