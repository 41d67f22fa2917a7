"""Paged mixed-width KV cache on the GPU.

A paged cache holds the same slots as the contiguous layout, only at other
addresses, and every kernel reads and writes it through the same slot order:
so the same appends and steps give bit-identical results on both.  Checked
for decode layer steps (a context fill per sequence, then two steps, some
pools crossing page ends), a two-layer decode stack (Sec. 3.3 and 3.8: one
pass, a cache per layer), read-back of whole pools, and the page accounting:
a sequence whose pages run out is dropped and flagged, a reset returns its
pages."""
import numpy as np
import pytest
import torch

import gen
import paper_2607_06601_amd as tr
from oracle.ties import enforce_margins
from paper_2607_06601_amd.device import DeviceLayer, to_dev

from _common import layer, npy
from test_gpu_layer import _taps, fill_context

pytestmark = pytest.mark.gpu
DEV = "cuda"
PT = 8  # tiles per page


def _pages(cfg, extra, slack=3):
    """Pages per width for the workload's context plus `extra` new tokens a
    sequence (enough whatever width the new tokens take)."""
    per = PT * (4096 // cfg["dh"])
    need = [slack] * 4
    for s in range(cfg["B"]):
        cnt = np.bincount(gen.context_bits(cfg, s), minlength=4)
        for bi in range(4):
            need[bi] += -(-(int(cnt[bi]) + extra) // per)
    return need


def _export(c, cache, s, bi, n, cfg):
    Hkv, dh, G = cfg["Hkv"], cfg["dh"], cfg["G"]
    if bi < 3:
        ko = torch.zeros(n, Hkv, dh, dtype=torch.uint8, device=DEV)
    else:
        ko = torch.zeros(n, Hkv, dh, dtype=torch.bfloat16, device=DEV)
    vo = torch.zeros_like(ko)
    ks = torch.zeros(n, Hkv, dh // G, 2, dtype=torch.int16, device=DEV)
    vs = torch.zeros_like(ks)
    pos = torch.zeros(n, dtype=torch.int32, device=DEV)
    tr.kv_export(c, cache, s, bi, 0, n, ko, vo, ks, vs, pos)
    return [ko, vo, ks, vs, pos]


@pytest.mark.parametrize("name", ["410m_bf16_decode", "1p3b_bf16_decode"])
def test_paged_decode_steps_equal_contiguous(name):
    L = layer(name)
    cfg = L["cfg"]
    D = DeviceLayer(L)
    c = D.cfg
    B, ctx = cfg["B"], cfg["ctx"]
    cont = tr.KVCache(c, B, ctx + 16)
    paged = tr.KVCache(c, B, ctx + 16, pages=(PT, _pages(cfg, 4)))
    print(f"paged {name}: {paged.nbytes / 2**20:.1f} MiB against {cont.nbytes / 2**20:.1f} MiB",
          flush=True)
    assert paged.nbytes < cont.nbytes / 2
    runs = []
    for cache in (cont, paged):
        fill_context(c, cache, cfg, D.act)
        x = D.x
        steps = []
        for _ in range(2):
            xo = torch.empty(B, cfg["d"], dtype=D.act, device=DEV)
            t, s = _taps(cfg, B, D.act)
            tr.layer_decode(c, B, x, D.psi, D.rw, D.dw, D.mw, cache, xo,
                            tr.workspace(c, tr.OP_LAYER_DECODE, B, 1), taps=s)
            steps.append((xo, t))
            x = xo
        torch.cuda.synchronize()
        assert cache.status() == 0
        runs.append(steps)
    for (xa, ta), (xb, tb) in zip(*runs):
        assert torch.equal(xa, xb)
        for n in ("o", "xt", "mode", "bit", "eidx"):
            assert torch.equal(ta[n], tb[n]), n
    assert torch.equal(cont.seq_len(), paged.seq_len())
    assert torch.equal(cont.pool_len(), paged.pool_len())
    lens = npy(cont.pool_len())
    for s in (0, B - 1):
        for bi in range(4):
            n = int(lens[s, bi])
            if n:
                for a, b in zip(_export(c, cont, s, bi, n, cfg), _export(c, paged, s, bi, n, cfg)):
                    assert torch.equal(a, b), (s, bi)
    free = paged.free_pages()
    held = [int(v) for v in paged.desc.n_pages]
    per = PT * (4096 // cfg["dh"])
    used = [int(sum(-(-int(lens[s, bi]) // per) for s in range(B))) for bi in range(4)]
    assert [h - f for h, f in zip(held, free)] == used


def test_paged_stack_equals_contiguous():
    Ls = gen.make_stack("410m_bf16_decode", 2)
    enforce_margins(Ls[0])
    cfg = Ls[0]["cfg"]
    Ds = [DeviceLayer(L) for L in Ls]
    c = Ds[0].cfg
    B = cfg["B"]
    outs = []
    for pages in (None, (PT, _pages(cfg, 2))):
        caches = []
        for D, L in zip(Ds, Ls):
            cache = tr.KVCache(D.cfg, B, cfg["ctx"] + 16, pages=pages)
            fill_context(D.cfg, cache, L["cfg"], D.act)
            caches.append(cache)
        xo = torch.empty(B, cfg["d"], dtype=Ds[0].act, device=DEV)
        tr.stack_decode(c, B, Ds[0].x, Ds[0].psi, [(D.rw, D.dw, D.mw) for D in Ds], caches, xo,
                        tr.workspace(c, tr.OP_STACK_DECODE, B, 1))
        torch.cuda.synchronize()
        assert all(ca.status() == 0 for ca in caches)
        outs.append((xo, [ca.pool_len().clone() for ca in caches]))
    assert torch.equal(outs[0][0], outs[1][0])
    for a, b in zip(outs[0][1], outs[1][1]):
        assert torch.equal(a, b)


def test_page_exhaustion_drops_the_row_and_reset_returns_pages():
    # d_h 64: 64-slot tiles; one tile per page; 2 pages of 2-bit, 1 of each other width
    c = tr.make_cfg(256, 4, 1, 64, 32, 4, 1, 512, 32, "bf16")
    cache = tr.KVCache(c, 3, 256, pages=(1, [2, 1, 1, 1]))
    assert cache.free_pages() == [2, 1, 1, 1]
    ws = tr.workspace(c, tr.OP_KV_APPEND, 1, 100)

    def append(seq, n, bi, tag):
        k, v = gen.kv_block(77, n, 1, 64, "bf16", 0.5, tag)
        tr.kv_append(c, cache, 1, n, to_dev(k.reshape(n, -1), torch.bfloat16),
                     to_dev(v.reshape(n, -1), torch.bfloat16),
                     torch.full((n,), bi, dtype=torch.uint8, device=DEV), ws,
                     seq_ids=torch.tensor([seq], dtype=torch.int32, device=DEV))
        torch.cuda.synchronize()

    append(0, 100, 0, "a")                     # two 2-bit pages
    assert cache.status() == 0 and cache.free_pages() == [0, 1, 1, 1]
    append(1, 10, 0, "b")                      # no 2-bit page left: dropped, flagged
    assert cache.status() & tr.CACHE_OVERFLOW
    assert int(cache.seq_len()[1]) == 0 and int(cache.pool_len()[1, 0]) == 0
    append(2, 5, 3, "c")                       # other widths still have pages
    assert int(cache.seq_len()[2]) == 5 and cache.free_pages() == [0, 1, 1, 0]
    cache.reset_seq(0)
    torch.cuda.synchronize()
    assert cache.free_pages() == [2, 1, 1, 0]
    assert int(cache.seq_len()[0]) == 0
    append(1, 10, 0, "b")                      # now it fits
    assert int(cache.seq_len()[1]) == 10 and cache.free_pages() == [1, 1, 1, 0]
