"""The no-allocation decode entry point (static device scratch) against
triroute_layer_decode with a caller workspace: identical inputs give
bit-identical outputs and caches, on two calls in a row, the second with a
smaller batch; an oversized batch is rejected before any launch."""
import ctypes as C

import numpy as np
import pytest
import torch

import gen
import paper_2607_06601_amd as tr
from paper_2607_06601_amd.device import DeviceLayer, to_dev

from _common import layer

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _fill(c, cache, cfg, ctx, act_t):
    ws = tr.workspace(c, tr.OP_KV_APPEND, 1, ctx)
    for s in range(cfg["B"]):
        k, v = gen.context_kv(cfg, s)
        bits = gen.context_bits(cfg, s)
        tr.kv_append(c, cache, 1, ctx, to_dev(k[:ctx].reshape(ctx, -1), act_t),
                     to_dev(v[:ctx].reshape(ctx, -1), act_t), to_dev(bits[:ctx], torch.uint8),
                     ws, seq_ids=torch.tensor([s], dtype=torch.int32, device=DEV))


def _taps(cfg, B, act_t):
    t = dict(o=torch.empty(B, cfg["H"] * cfg["dh"], dtype=act_t, device=DEV),
             xt=torch.empty(B, cfg["d"], dtype=act_t, device=DEV),
             mode=torch.empty(B, cfg["H"], dtype=torch.uint8, device=DEV))
    return t, tr.Taps(**{n: x.data_ptr() for n, x in t.items()})


@pytest.mark.parametrize("name", ["410m_bf16_decode", "1p3b_bf16_decode"])
def test_noalloc_decode_matches_workspace_decode(name):
    L = layer(name)
    cfg = L["cfg"]
    D = DeviceLayer(L)
    c = D.cfg
    ctx = 1500
    caches = [tr.KVCache(c, cfg["B"], ctx + 8) for _ in range(2)]
    for cache in caches:
        _fill(c, cache, cfg, ctx, D.act)
    torch.cuda.synchronize()
    for B in (cfg["B"], cfg["B"] // 4):          # the second call on a smaller batch
        sid = to_dev(np.arange(B, dtype=np.int32)[::-1].copy(), torch.int32)
        x, psi = D.x[:B].contiguous(), D.psi[:B].contiguous()
        out = []
        for path, cache in zip(("workspace", "static"), caches):
            xo = torch.empty(B, cfg["d"], dtype=D.act, device=DEV)
            t, taps = _taps(cfg, B, D.act)
            if path == "workspace":
                ws = tr.workspace(c, tr.OP_LAYER_DECODE, B, 1)
                tr.layer_decode(c, B, x, psi, D.rw, D.dw, D.mw, cache, xo, ws, taps=taps,
                                seq_ids=sid)
            else:
                tr.layer_decode_noalloc(c, B, x, psi, D.rw, D.dw, D.mw, cache, xo, taps=taps,
                                        seq_ids=sid)
            torch.cuda.synchronize()
            assert cache.status() == 0
            out.append((xo, t))
        (xa, ta), (xb, tb) = out
        assert torch.equal(xa, xb), f"x_out differs at B={B}"
        for n in ta:
            assert torch.equal(ta[n], tb[n]), f"{n} differs at B={B}"
        assert torch.equal(caches[0].buf, caches[1].buf), f"cache differs at B={B}"


def test_noalloc_rejects_a_batch_beyond_the_static_scratch():
    c = tr.make_cfg(2048, 16, 4, 128, 1024, 16, 2, 5632, 64, "bf16")
    need = tr.workspace_bytes(c, tr.OP_LAYER_DECODE, 512, 1)
    assert need > 16 << 20
    fake = 1 << 40
    rw = tr.RouterW(*([fake] * 12))
    dw = tr.DenseW(*([fake] * 5))
    mw = tr.MoeW(*([fake] * 3))
    desc = tr.KVCacheDesc()
    r = tr.lib().triroute_layer_decode_noalloc(C.byref(c), 512, None, fake, fake, C.byref(rw),
                                               C.byref(dw), C.byref(mw), C.byref(desc), fake,
                                               None, None)
    assert r == -3 and b"static" in tr.lib().triroute_last_error()
