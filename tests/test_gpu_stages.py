"""Per-stage parity of the HIP path against the CPU oracle (through the C ABI).

Discrete results (routing decisions, compaction lists, KV codes, scales,
positions) must be bit exact; activations within the bf16 / fp32 tolerance.
Every input comes from the seeded generator; the oracle never sees a value
the GPU produced."""
import numpy as np
import pytest
import torch

import gen
import oracle
import paper_2607_06601_amd as tr
from oracle import quant
from paper_2607_06601_amd.device import DeviceLayer, cfg_from, to_dev

from _common import assert_close, layer, note, npy, shape_of, torch_act

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tr.lib()
    yield
    torch.cuda.synchronize()


# ------------------------------------------------------------------ router
def run_router(L):
    cfg = L["cfg"]
    D = DeviceLayer(L, moe=False)
    c = D.cfg
    B, T, H, k = cfg["B"], cfg["T"], cfg["H"], cfg["k"]
    N = B * T
    n1 = torch.empty(N, cfg["d"], dtype=D.act, device=DEV)
    mode = torch.empty(N, H, dtype=torch.uint8, device=DEV)
    bit = torch.empty(N, dtype=torch.uint8, device=DEV)
    eidx = torch.empty(N, k, dtype=torch.int32, device=DEV)
    egate = torch.empty(N, k, dtype=torch.float32, device=DEV)
    cmp = tr.CompactionBuffers(c, B, T)
    ws = tr.workspace(c, tr.OP_ROUTER, B, T)
    tr.router(c, B, T, D.x, D.psi, D.rw, n1, mode, bit, eidx, egate, cmp.struct, ws)
    torch.cuda.synchronize()
    return dict(n1=n1, mode=mode, bit=bit, eidx=eidx, egate=egate, cmp=cmp)


@pytest.mark.parametrize("name,seed,groups", [
    ("tiny_f32_prefill", 0, None), ("160m_bf16_prefill", 1, None), ("410m_bf16_decode", 103, None),
    ("1p3b_bf16_prefill", 104, None), ("1p3b_bf16_decode", 105, None),
    # attention decisions per token / per kv-head group instead of per head
    ("160m_bf16_prefill", 1, 1), ("1p3b_bf16_decode", 105, 4)])
def test_router_and_compaction_bit_exact(name, seed, groups):
    L = layer(name, seed, moe=False)
    if groups is not None:
        L = gen.granularity_variant(L, groups)
    cfg = L["cfg"]
    B, T, H, E, k = cfg["B"], cfg["T"], cfg["H"], cfg["E"], cfg["k"]
    g = run_router(L)
    n1, za, ze, zb = oracle.router_logits(L)
    mode, bit, eidx, egate = oracle.decide(za, ze, zb, k, H)
    if groups is not None:
        R = H // groups
        assert all((mode[:, a * R:(a + 1) * R] == mode[:, a * R:a * R + 1]).all()
                   for a in range(groups))
    np.testing.assert_array_equal(npy(g["mode"]), mode)
    np.testing.assert_array_equal(npy(g["bit"]), bit)
    np.testing.assert_array_equal(npy(g["eidx"]), eidx)
    np.testing.assert_allclose(npy(g["egate"]), egate, rtol=2e-5, atol=1e-6)
    assert_close(npy(g["n1"]), oracle.layer.to_native(n1, cfg["act"]) if cfg["act"] == "f32"
                 else n1, cfg["act"], "n1")
    c = oracle.compact(mode, eidx, B, T, H, E, k)
    cnt = npy(g["cmp"].attn_cnt)
    np.testing.assert_array_equal(cnt, c["attn_cnt"])
    idx = npy(g["cmp"].attn_idx).reshape(B * H * 2, T)
    for s in range(B * H * 2):
        np.testing.assert_array_equal(idx[s, :cnt[s]], c["attn_idx"][s, :cnt[s]])
    np.testing.assert_array_equal(npy(g["cmp"].exp_cnt), c["exp_cnt"])
    np.testing.assert_array_equal(npy(g["cmp"].exp_off), c["exp_off"])
    nreal = int(c["exp_off"][-1])
    np.testing.assert_array_equal(npy(g["cmp"].exp_rows)[:nreal], c["exp_rows"])


# ------------------------------------------------------------ KV append
KV_SHAPES = [  # (act, dh, G, Hkv)
    ("f32", 64, 32, 1), ("bf16", 64, 64, 3), ("bf16", 128, 64, 4), ("bf16", 128, 32, 2)]


def kv_cfg(act, dh, G, Hkv):
    return tr.make_cfg(256, 4 * Hkv, Hkv, dh, 32, 4, 1, 512, G, act)


def export_pool(c, cache, s, bi, n, act, Hkv, dh, G):
    tdt = torch_act(act)
    if bi < 3:
        ko = torch.zeros(n, Hkv, dh, dtype=torch.uint8, device=DEV)
        vo = torch.zeros_like(ko)
    else:
        ko = torch.zeros(n, Hkv, dh, dtype=tdt, device=DEV)
        vo = torch.zeros_like(ko)
    ks = torch.zeros(n, Hkv, dh // G, 2, dtype=torch.int16, device=DEV)
    vs = torch.zeros_like(ks)
    pos = torch.zeros(n, dtype=torch.int32, device=DEV)
    tr.kv_export(c, cache, s, bi, 0, n, ko, vo, ks, vs, pos)
    torch.cuda.synchronize()
    return ko, vo, ks, vs, pos


def _f16(bits_i16):
    return np.asarray(bits_i16).astype(np.int16).view(np.float16)


@pytest.mark.parametrize("act,dh,G,Hkv", KV_SHAPES)
def test_kv_append_codes_bit_exact(act, dh, G, Hkv):
    B, T1, T2, cap = 3, 37, 58, 200
    c = kv_cfg(act, dh, G, Hkv)
    tdt = torch_act(act)
    k, v = gen.kv_block(11, B * (T1 + T2), Hkv, dh, act, std=0.7)
    k, v = k.reshape(B, T1 + T2, Hkv, dh), v.reshape(B, T1 + T2, Hkv, dh)
    bits = gen.stream(11, "kvbits").integers(0, 4, (B, T1 + T2)).astype(np.uint8)
    cache = tr.KVCache(c, B + 1, cap)
    for (t0, t1) in ((0, T1), (T1, T1 + T2)):
        Tn = t1 - t0
        kd = to_dev(k[:, t0:t1].reshape(B * Tn, Hkv * dh), tdt)
        vd = to_dev(v[:, t0:t1].reshape(B * Tn, Hkv * dh), tdt)
        bd = to_dev(bits[:, t0:t1].reshape(-1), torch.uint8)
        sid = torch.tensor([2, 0, 1], dtype=torch.int32, device=DEV)
        ws = tr.workspace(c, tr.OP_KV_APPEND, B, Tn)
        tr.kv_append(c, cache, B, Tn, kd, vd, bd, ws, seq_ids=sid)
    torch.cuda.synchronize()
    assert cache.status() == 0
    seq_of_row = [2, 0, 1]
    np.testing.assert_array_equal(npy(cache.seq_len())[[2, 0, 1, 3]], [T1 + T2] * 3 + [0])
    for b in range(B):
        s = seq_of_row[b]
        for bi, nb in enumerate(quant.BITS):
            toks = np.flatnonzero(bits[b] == bi)
            assert int(npy(cache.pool_len())[s, bi]) == len(toks)
            if len(toks) == 0:
                continue
            ko, vo, ks, vs, pos = export_pool(c, cache, s, bi, len(toks), act, Hkv, dh, G)
            np.testing.assert_array_equal(npy(pos), toks)
            for src, out, sz in ((k, ko, ks), (v, vo, vs)):
                x = src[b, toks]
                if nb == 16:
                    np.testing.assert_array_equal(npy(out).astype(np.float32), x)
                    continue
                codes, s16, z16 = quant.quantize(x, nb, G)
                np.testing.assert_array_equal(npy(out), codes)
                szn = npy(sz)
                np.testing.assert_array_equal(_f16(szn[..., 0]).view(np.uint16), s16.view(np.uint16))
                np.testing.assert_array_equal(_f16(szn[..., 1]).view(np.uint16), z16.view(np.uint16))


def _host_decode(raw: np.ndarray, desc, c, s, bi, g, slot, ch, isv, act):
    """Independent reading of the documented physical layout (include/triroute.h)."""
    dh, Hkv = c.head_dim, c.n_kv_heads
    bp = [2, 4, 8, 16 if act == "bf16" else 32][bi]
    TS = 4096 // dh
    tile, st = divmod(slot, TS)
    base = desc.off_pool[bi] + ((s * Hkv + g) * desc.n_tiles + tile) * desc.tile_bytes[bi]
    if isv:
        base += 512 * bp
        r = st % 32
        f = (st // 32) * (dh // 16) + ch // 16
        lane = ((r % 16) // 4) * 16 + ch % 16
        j = (r // 16) * 4 + r % 4
    else:
        f = (st // 16) * (dh // 32) + ch // 32
        lane = ((ch % 32) // 8) * 16 + st % 16
        j = ch % 8
    q = f * 8 + j
    rec = base + lane * 8 * bp
    if bp == 32:
        return int(raw[rec + 4 * q: rec + 4 * q + 4].view(np.uint32)[0])
    f, j = q // 8, q % 8
    if bp == 2:
        word, bitpos = q // 16, 4 * j + 2 * (f % 2)
    elif bp == 4:
        word, bitpos = q // 8, 8 * (j % 4) + 4 * (j // 4)
    elif bp == 8:
        word, bitpos = q // 4, 8 * (q % 4)
    else:
        word, bitpos = q // 2, 16 * (q % 2)
    w = int(raw[rec + 4 * word: rec + 4 * word + 4].view(np.uint32)[0])
    return (w >> bitpos) & ((1 << bp) - 1)


@pytest.mark.parametrize("act,dh,G,Hkv", KV_SHAPES[:3])
def test_kv_physical_layout_matches_header(act, dh, G, Hkv):
    c = kv_cfg(act, dh, G, Hkv)
    n = 70
    k, v = gen.kv_block(12, n, Hkv, dh, act)
    bits = gen.stream(12, "kvbits").integers(0, 4, n).astype(np.uint8)
    cache = tr.KVCache(c, 1, 128)
    tdt = torch_act(act)
    tr.kv_append(c, cache, 1, n, to_dev(k.reshape(n, -1), tdt), to_dev(v.reshape(n, -1), tdt),
                 to_dev(bits, torch.uint8), tr.workspace(c, tr.OP_KV_APPEND, 1, n))
    torch.cuda.synchronize()
    raw = cache.buf.cpu().numpy()
    rng = np.random.default_rng(0)
    for bi in range(4):
        m = int((bits == bi).sum())
        if m == 0:
            continue
        ko, vo, _, _, _ = export_pool(c, cache, 0, bi, m, act, Hkv, dh, G)
        kon, von = npy(ko), npy(vo)
        if bi == 3:
            kon = kon.astype(np.float32).view(np.uint32) >> (16 if act == "bf16" else 0)
            von = von.astype(np.float32).view(np.uint32) >> (16 if act == "bf16" else 0)
        for _ in range(40):
            slot, g, ch = int(rng.integers(m)), int(rng.integers(Hkv)), int(rng.integers(dh))
            assert _host_decode(raw, cache.desc, c, 0, bi, g, slot, ch, False, act) == kon[slot, g, ch]
            assert _host_decode(raw, cache.desc, c, 0, bi, g, slot, ch, True, act) == von[slot, g, ch]


def test_kv_capacity_overflow_sets_flag_and_drops_row():
    c = kv_cfg("bf16", 64, 64, 1)
    cache = tr.KVCache(c, 2, 16)
    k, v = gen.kv_block(13, 2 * 10, 1, 64, "bf16")
    kd, vd = to_dev(k.reshape(20, -1), torch.bfloat16), to_dev(v.reshape(20, -1), torch.bfloat16)
    bd = torch.zeros(20, dtype=torch.uint8, device=DEV)
    ws = tr.workspace(c, tr.OP_KV_APPEND, 2, 10)
    tr.kv_append(c, cache, 2, 10, kd, vd, bd, ws)
    assert cache.status() == 0
    tr.kv_append(c, cache, 2, 10, kd, vd, bd, ws)     # 20 > 16: both rows dropped
    assert cache.status() == tr.CACHE_OVERFLOW
    np.testing.assert_array_equal(npy(cache.seq_len()), [10, 10])
    with pytest.raises(tr.TrirouteError):              # host-visible: T > capacity
        tr.kv_append(c, cache, 1, 17, kd, vd, bd, tr.workspace(c, tr.OP_KV_APPEND, 1, 17))


# ------------------------------------------------------------------- QKV
# T 133: few-token tiles (ragged against 32-row tiles); T 1500 / 1100: the
# many-token four-wave path (ragged against 256-row tiles)
@pytest.mark.parametrize("name,T", [("tiny_f32_prefill", 133), ("160m_bf16_prefill", 133),
                                    ("1p3b_bf16_prefill", 133), ("160m_bf16_prefill", 1500),
                                    ("1p3b_bf16_prefill", 1100)])
def test_qkv_rope(name, T):
    L = gen.make_layer(name, with_moe=False)
    cfg = L["cfg"]
    act = cfg["act"]
    B = 2
    x = gen.to_act(gen.normal(41, "qkv_in", (B * T, cfg["d"])), act)
    D = DeviceLayer(L, moe=False)
    c = D.cfg
    H, Hkv, dh = cfg["H"], cfg["Hkv"], cfg["dh"]
    pos0 = np.array([0, 30000], np.int32)               # long positions stress RoPE angles
    n1 = to_dev(x, D.act)
    q = torch.empty(B * T, H * dh, dtype=D.act, device=DEV)
    k = torch.empty(B * T, Hkv * dh, dtype=D.act, device=DEV)
    v = torch.empty_like(k)
    ws = tr.workspace(c, tr.OP_QKV, B, T)
    tr.qkv(c, B, T, n1, D.dw, q, k, v, ws, pos0=to_dev(pos0, torch.int32))
    torch.cuda.synchronize()
    pos = np.concatenate([p + np.arange(T) for p in pos0])
    qo, ko, vo = oracle.qkv(np.asarray(x, np.float64), L, pos)
    assert_close(npy(q), qo.reshape(B * T, -1), act, "q")
    assert_close(npy(k), ko.reshape(B * T, -1), act, "k")
    assert_close(npy(v), vo.reshape(B * T, -1), act, "v")


# ------------------------------------------------------------- attention
def _fill_cache(c, cache, kk, vv, bits, act, seq_ids=None):
    B, T = bits.shape
    tdt = torch_act(act)
    tr.kv_append(c, cache, B, T, to_dev(kk.reshape(B * T, -1), tdt),
                 to_dev(vv.reshape(B * T, -1), tdt), to_dev(bits.reshape(-1), torch.uint8),
                 tr.workspace(c, tr.OP_KV_APPEND, B, T),
                 seq_ids=None if seq_ids is None else to_dev(np.asarray(seq_ids, np.int32), torch.int32))


ATTN_SHAPES = [  # (act, H, Hkv, dh, G, w, B, T, ctx): T queries after ctx cached tokens
    ("f32", 4, 1, 64, 32, 32, 1, 128, 0),
    ("bf16", 12, 3, 64, 64, 48, 2, 150, 0),
    ("bf16", 16, 4, 128, 64, 40, 2, 97, 0),
    ("bf16", 16, 2, 64, 32, 64, 2, 200, 300),    # 8 heads per kv head: two quartets
    ("bf16", 6, 3, 128, 32, 50, 2, 120, 0),      # 2 heads per kv head: half quartets
    ("bf16", 16, 4, 128, 64, 100, 3, 160, 1000),  # long cached context
]


@pytest.mark.parametrize("act,H,Hkv,dh,G,w,B,T,ctx", ATTN_SHAPES)
def test_attention_prefill(act, H, Hkv, dh, G, w, B, T, ctx):
    c = tr.make_cfg(256, H, Hkv, dh, w, 4, 1, 512, G, act)
    std = 0.6
    P = ctx + T
    kk, vv = gen.kv_block(21, B * P, Hkv, dh, act, std)
    kk, vv = kk.reshape(B, P, Hkv, dh), vv.reshape(B, P, Hkv, dh)
    qq = gen.to_act(gen.normal(21, "attn_q", (B, T, H, dh), std), act)
    rng = gen.stream(21, "attn_modes")
    modes = rng.choice(3, size=(B * T, H), p=[0.25, 0.45, 0.30]).astype(np.uint8)
    bits = rng.integers(0, 4, (B, P)).astype(np.uint8)
    cache = tr.KVCache(c, B, P + 8)
    _fill_cache(c, cache, kk, vv, bits, act)
    cm = oracle.compact(modes, np.zeros((B * T, 1), np.int32), B, T, H, 4, 1)
    cmp = tr.CompactionBuffers(c, B, T)
    cmp.attn_cnt.copy_(to_dev(cm["attn_cnt"], torch.int32))
    cmp.attn_idx.copy_(to_dev(np.where(cm["attn_idx"] < 0, 0, cm["attn_idx"]).reshape(-1), torch.int32))
    o = torch.empty(B * T, H * dh, dtype=torch_act(act), device=DEV)
    qd = to_dev(qq.reshape(B * T, H * dh), torch_act(act))
    md = to_dev(modes, torch.uint8)
    tr.attn_prefill(c, B, T, qd, cache, md, cmp.struct, o,
                    ws=tr.workspace(c, tr.OP_ATTN_PREFILL, B, T))
    torch.cuda.synchronize()
    og = npy(o).reshape(B, T, H, dh)
    cfgd = dict(G=G)
    for b in range(B):
        khat, vhat, _ = oracle.layer.store_kv(kk[b], vv[b], bits[b], cfgd)
        ref = oracle.attention_seq(np.asarray(qq[b], np.float64), ctx + np.arange(T), khat, vhat,
                                   modes[b * T:(b + 1) * T], w)
        assert_close(og[b], ref, act, f"o[b={b}]")


@pytest.mark.parametrize("act,H,Hkv,dh,G,w,ctx,B", [
    ("f32", 4, 1, 64, 32, 32, 300, 5),
    ("bf16", 16, 4, 64, 64, 256, 1500, 5),        # 4 heads per kv head, split into chunks
    ("bf16", 16, 4, 128, 64, 100, 2100, 5),
    ("bf16", 16, 2, 64, 32, 64, 700, 5),          # 8 heads per kv head: one head per column
    ("bf16", 6, 3, 128, 32, 50, 900, 5),          # 2 heads per kv head
    ("bf16", 8, 4, 64, 64, 96, 260, 64),          # one chunk per (sequence, kv head)
])
def test_attention_decode(act, H, Hkv, dh, G, w, ctx, B):
    c = tr.make_cfg(256, H, Hkv, dh, w, 4, 1, 512, G, act)
    kk, vv = gen.kv_block(22, B * (ctx + 1), Hkv, dh, act, 0.8)
    kk, vv = kk.reshape(B, ctx + 1, Hkv, dh), vv.reshape(B, ctx + 1, Hkv, dh)
    rng = gen.stream(22, "dec")
    bits = rng.integers(0, 4, (B, ctx + 1)).astype(np.uint8)
    modes = rng.choice(3, size=(B, H), p=[0.2, 0.4, 0.4]).astype(np.uint8)
    modes[0] = 0                                          # a sequence whose heads all skip
    modes[1] = 1                                          # all local
    modes[2, 0] = 2                                       # mixed modes within a kv head
    modes[2, 1:] = 0
    qq = gen.to_act(gen.normal(22, "dec_q", (B, H, dh), 0.8), act)
    cache = tr.KVCache(c, B, ctx + 4)
    # context in two appends (ragged), then the new token
    _fill_cache(c, cache, kk[:, :ctx // 2], vv[:, :ctx // 2], bits[:, :ctx // 2], act)
    _fill_cache(c, cache, kk[:, ctx // 2:ctx], vv[:, ctx // 2:ctx], bits[:, ctx // 2:ctx], act)
    _fill_cache(c, cache, kk[:, ctx:], vv[:, ctx:], bits[:, ctx:], act)
    o = torch.empty(B, H * dh, dtype=torch_act(act), device=DEV)
    tr.attn_decode(c, B, to_dev(qq.reshape(B, -1), torch_act(act)), cache,
                   to_dev(modes, torch.uint8), o, ws=tr.workspace(c, tr.OP_ATTN_DECODE, B, 1))
    torch.cuda.synchronize()
    og = npy(o).reshape(B, H, dh)
    cfgd = dict(G=G)
    for b in range(B):
        khat, vhat, _ = oracle.layer.store_kv(kk[b], vv[b], bits[b], cfgd)
        ref = oracle.attention_seq(np.asarray(qq[b:b + 1], np.float64), np.array([ctx]), khat,
                                   vhat, modes[b:b + 1], w)[0]
        assert_close(og[b], ref, act, f"o[b={b}]")
    assert not og[0].any()


# ------------------------------------------------------------ O-proj, MoE
@pytest.mark.parametrize("name,n_tok", [("tiny_f32_prefill", 128), ("160m_bf16_prefill", 301),
                                        ("1p3b_bf16_decode", 32)])
def test_oproj_and_moe(name, n_tok):
    L = gen.make_layer(name)
    cfg = L["cfg"]
    act, H, dh, d, E, k = cfg["act"], cfg["H"], cfg["dh"], cfg["d"], cfg["E"], cfg["k"]
    D = DeviceLayer(L)
    c = D.cfg
    x = L["x"][:n_tok]
    o = gen.to_act(gen.normal(31, "o_in", (n_tok, H * dh), 0.5), act)
    xt = torch.empty(n_tok, d, dtype=D.act, device=DEV)
    tr.oproj(c, n_tok, to_dev(x, D.act), to_dev(o, D.act), D.dw, xt)
    torch.cuda.synchronize()
    ref_xt = oracle.oproj(x, np.asarray(o, np.float64), L["Wo"])
    assert_close(npy(xt), ref_xt, act, "xt")
    # experts on a generator-made xt with decisions from random logits
    xt_in = gen.to_act(gen.normal(32, "xt_in", (n_tok, d)), act)
    ze = gen.normal(32, "ze", (n_tok, E + 1), 1.5).astype(np.float64)
    _, _, eidx, egate = oracle.decide(np.zeros((n_tok, 1, 3)), ze, np.zeros((n_tok, 4)), k)
    cm = oracle.compact(np.zeros((n_tok, 1), np.uint8), eidx, n_tok, 1, 1, E, k)
    cmp = tr.CompactionBuffers(c, n_tok, 1)
    cmp.exp_cnt.copy_(to_dev(cm["exp_cnt"], torch.int32))
    cmp.exp_off.copy_(to_dev(cm["exp_off"], torch.int32))
    cmp.exp_rows[:len(cm["exp_rows"])].copy_(to_dev(cm["exp_rows"], torch.int32))
    xo = torch.empty(n_tok, d, dtype=D.act, device=DEV)
    tr.moe(c, n_tok, to_dev(xt_in, D.act), D.dw, D.mw, to_dev(eidx, torch.int32),
           to_dev(egate.astype(np.float32), torch.float32), cmp.struct, xo,
           tr.workspace(c, tr.OP_MOE, n_tok, 1))
    torch.cuda.synchronize()
    ref, _, _ = oracle.moe(np.asarray(xt_in, np.float64), L, eidx, egate.astype(np.float32))
    assert_close(npy(xo), ref, act, "x_out")
    null_only = np.all(eidx == 0, axis=1)
    np.testing.assert_array_equal(npy(xo)[null_only], xt_in[null_only])


def test_kv_reset_and_reuse_overwrites_slots():
    """After reset_seq, new appends land on the same slots and fully replace
    the previous contents (sub-byte V words included)."""
    act, dh, G, Hkv = "bf16", 64, 64, 2
    c = kv_cfg(act, dh, G, Hkv)
    n = 90
    cache = tr.KVCache(c, 1, 128)
    bits = gen.stream(14, "kvbits").integers(0, 4, n).astype(np.uint8)
    for rep, seed in enumerate((14, 15)):
        if rep:
            cache.reset_seq(0)
        k, v = gen.kv_block(seed, n, Hkv, dh, act)
        tr.kv_append(c, cache, 1, n, to_dev(k.reshape(n, -1), torch.bfloat16),
                     to_dev(v.reshape(n, -1), torch.bfloat16), to_dev(bits, torch.uint8),
                     tr.workspace(c, tr.OP_KV_APPEND, 1, n))
    torch.cuda.synchronize()
    for bi, nb in enumerate(quant.BITS):
        toks = np.flatnonzero(bits == bi)
        if len(toks) == 0:
            continue
        ko, vo, _, _, _ = export_pool(c, cache, 0, bi, len(toks), act, Hkv, dh, G)
        for src, out in ((k, ko), (v, vo)):
            if nb == 16:
                np.testing.assert_array_equal(npy(out).astype(np.float32), src[toks])
            else:
                np.testing.assert_array_equal(npy(out), quant.quantize(src[toks], nb, G)[0])


# ----------------------------------------- single-token appends (decode)
@pytest.mark.parametrize("act,dh,G,Hkv", [("bf16", 64, 64, 4), ("bf16", 128, 64, 4),
                                          ("bf16", 64, 32, 2), ("f32", 64, 32, 1)])
def test_kv_append_one_token_rows_bit_exact(act, dh, G, Hkv):
    """The decode append (one token per row, 2/4-bit V codes set in words
    shared with earlier slots): 64 rows with different starting lengths,
    then 40 one-token appends; every slot of every pool equals the oracle's
    quantization of the token it holds (paper Sec. 3.2 (C))."""
    B, steps = 64, 40
    c = kv_cfg(act, dh, G, Hkv)
    tdt = torch_act(act)
    start = np.array([(7 * r) % 37 for r in range(B)])
    total = start + steps
    k, v = gen.kv_block(16, B * int(total.max()), Hkv, dh, act, std=0.9)
    k = k.reshape(B, -1, Hkv, dh)
    v = v.reshape(B, -1, Hkv, dh)
    bits = gen.stream(16, "kvbits1").integers(0, 4, (B, int(total.max()))).astype(np.uint8)
    cache = tr.KVCache(c, B + 2, int(total.max()) + 8)
    seq_of = gen.stream(16, "seqperm").permutation(B + 2)[:B].astype(np.int32)
    for r in range(B):          # starting lengths, one row per call
        n = int(start[r])
        if n == 0:
            continue
        tr.kv_append(c, cache, 1, n, to_dev(k[r, :n].reshape(n, -1), tdt),
                     to_dev(v[r, :n].reshape(n, -1), tdt), to_dev(bits[r, :n], torch.uint8),
                     tr.workspace(c, tr.OP_KV_APPEND, 1, n),
                     seq_ids=to_dev(seq_of[r:r + 1], torch.int32))
    sid = to_dev(seq_of, torch.int32)
    ws = tr.workspace(c, tr.OP_KV_APPEND, B, 1)
    for j in range(steps):      # one new token per row, at each row's own position
        t_idx = start + j
        kd = to_dev(k[np.arange(B), t_idx].reshape(B, -1), tdt)
        vd = to_dev(v[np.arange(B), t_idx].reshape(B, -1), tdt)
        bd = to_dev(bits[np.arange(B), t_idx], torch.uint8)
        tr.kv_append(c, cache, B, 1, kd, vd, bd, ws, seq_ids=sid)
    torch.cuda.synchronize()
    assert cache.status() == 0
    np.testing.assert_array_equal(npy(cache.seq_len())[seq_of], total)
    for r in range(B):
        s_ = int(seq_of[r])
        n = int(total[r])
        for bi, nb in enumerate(quant.BITS):
            toks = np.flatnonzero(bits[r, :n] == bi)
            assert int(npy(cache.pool_len())[s_, bi]) == len(toks)
            if len(toks) == 0:
                continue
            ko, vo, ks, vs, pos = export_pool(c, cache, s_, bi, len(toks), act, Hkv, dh, G)
            np.testing.assert_array_equal(npy(pos), toks)
            for src, out, sz in ((k, ko, ks), (v, vo, vs)):
                x = src[r, toks]
                if nb == 16:
                    np.testing.assert_array_equal(npy(out).astype(np.float32), x)
                    continue
                codes, s16, z16 = quant.quantize(x, nb, G)
                np.testing.assert_array_equal(npy(out), codes)
                szn = npy(sz)
                np.testing.assert_array_equal(_f16(szn[..., 0]).view(np.uint16), s16.view(np.uint16))
                np.testing.assert_array_equal(_f16(szn[..., 1]).view(np.uint16), z16.view(np.uint16))


def test_layer_prefill_bad_sequence_id_is_flagged():
    """A row naming a sequence outside the cache is dropped by the append,
    sets TRIROUTE_CACHE_BAD_SEQ, and reads no position out of bounds: its
    outputs stay finite and the other rows are unaffected."""
    L = layer("tiny_f32_prefill", 0)
    L["cfg"]["B"], L["cfg"]["T"] = 2, 64
    L["x"] = np.concatenate([L["x"][:64], L["x"][64:128]])
    D = DeviceLayer(L)
    c = D.cfg
    cache = tr.KVCache(c, 2, 64)
    xo = torch.empty(128, L["cfg"]["d"], dtype=D.act, device=DEV)
    ws = tr.workspace(c, tr.OP_LAYER_PREFILL, 2, 64)
    sid = torch.tensor([0, 2], dtype=torch.int32, device=DEV)    # 2 == n_seq
    tr.layer_prefill(c, 2, 64, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo, ws, seq_ids=sid)
    torch.cuda.synchronize()
    assert cache.status() == tr.CACHE_BAD_SEQ
    assert torch.isfinite(xo).all()
    np.testing.assert_array_equal(npy(cache.seq_len()), [64, 0])


# ----------------------------------------------- full-size expert block
def _moe_case(L, n_tok, eidx, egate, tag):
    """triroute_moe on a generator-made x~ with the given routing, every row
    against the oracle's expert block (paper Sec. 3.2 (B) expert equation)."""
    cfg = L["cfg"]
    act, d, E, k = cfg["act"], cfg["d"], cfg["E"], cfg["k"]
    D = DeviceLayer(L)
    c = D.cfg
    xt_in = gen.to_act(gen.normal(33, "xt_full", (n_tok, d)), act)
    cm = oracle.compact(np.zeros((n_tok, 1), np.uint8), eidx, n_tok, 1, 1, E, k)
    cmp = tr.CompactionBuffers(c, n_tok, 1)
    cmp.exp_cnt.copy_(to_dev(cm["exp_cnt"], torch.int32))
    cmp.exp_off.copy_(to_dev(cm["exp_off"], torch.int32))
    if len(cm["exp_rows"]):
        cmp.exp_rows[:len(cm["exp_rows"])].copy_(to_dev(cm["exp_rows"], torch.int32))
    xo = torch.empty(n_tok, d, dtype=D.act, device=DEV)
    tr.moe(c, n_tok, to_dev(xt_in, D.act), D.dw, D.mw, to_dev(eidx, torch.int32),
           to_dev(egate.astype(np.float32), torch.float32), cmp.struct, xo,
           tr.workspace(c, tr.OP_MOE, n_tok, 1))
    torch.cuda.synchronize()
    del D
    ref, _, _ = oracle.moe(np.asarray(xt_in, np.float64), L, eidx,
                           egate.astype(np.float32).astype(np.float64))
    assert_close(npy(xo), ref, act, f"x_out ({tag})")
    null_only = np.all(eidx == 0, axis=1)
    np.testing.assert_array_equal(npy(xo)[null_only], xt_in[null_only])
    return cm


@pytest.mark.parametrize("name", ["160m_bf16_prefill", "1p3b_bf16_prefill"])
def test_moe_and_oproj_full_size(name):
    """The many-token grouped GEMMs and O-projection at the workload's own
    token count (B*T = 16384, > 2048 assignments), every row."""
    L = gen.make_layer(name)
    cfg = L["cfg"]
    act, H, dh, E, k = cfg["act"], cfg["H"], cfg["dh"], cfg["E"], cfg["k"]
    N = cfg["B"] * cfg["T"]
    D = DeviceLayer(L, moe=False)
    o = gen.to_act(gen.normal(34, "o_full", (N, H * dh), 0.5), act)
    xt = torch.empty(N, cfg["d"], dtype=D.act, device=DEV)
    tr.oproj(D.cfg, N, D.x, to_dev(o, D.act), D.dw, xt)
    torch.cuda.synchronize()
    assert_close(npy(xt), oracle.oproj(L["x"], np.asarray(o, np.float64), L["Wo"]), act,
                 "x~ (oproj, many-token)")
    del D, xt
    ze = gen.normal(35, "ze_full", (N, E + 1), 1.5).astype(np.float64)
    _, _, eidx, egate = oracle.decide(np.zeros((N, 1, 3)), ze, np.zeros((N, 4)), k)
    cm = _moe_case(L, N, eidx, egate, "uniform, many-token")
    assert cm["exp_off"][-1] > 2048


def _routing_with_counts(counts, n_both_null, N, k, seed):
    """eidx [N, 2] / egate with exactly counts[e] assignments to expert e
    (index 0: null slots outside the both-null tokens), n_both_null tokens
    whose two slots are both null, ids ascending within a token, rows in a
    seeded random order."""
    assert k == 2
    rest = N - n_both_null
    ids = np.repeat(np.arange(len(counts)), counts)
    assert len(ids) == 2 * rest and max(counts) <= rest
    pairs = np.stack([ids[:rest], ids[rest:]], axis=1)       # sorted: distinct, ascending
    pairs = np.concatenate([np.zeros((n_both_null, 2), np.int64), pairs])
    g = gen.stream(seed, "perm")
    pairs = pairs[g.permutation(N)].astype(np.int32)
    w = g.random((N, 2)) + 0.05
    egate = w / w.sum(axis=1, keepdims=True)
    egate[pairs == 0] *= 0.5                                   # the null's share is dropped
    return pairs, egate


def test_moe_expert_count_edges():
    """Expert lists of 0, 1, 255, 256, 257, 511 and 513 rows (tile edges of
    the 256-row tiles), tokens with both slots null, > 2048 assignments."""
    L = gen.make_layer("160m_bf16_prefill")
    N, E = 1300, L["cfg"]["E"]
    nb = 9
    counts = [120, 0, 1, 255, 256, 257, 511, 513]
    counts.append(2 * (N - nb) - sum(counts))
    eidx, egate = _routing_with_counts(np.array(counts), nb, N, 2, 36)
    cm = _moe_case(L, N, eidx, egate, "count edges")
    np.testing.assert_array_equal(cm["exp_cnt"][1:], counts[1:])
    assert (np.all(eidx == 0, axis=1)).sum() == nb


def test_moe_skewed_prefill_scale():
    """Skewed routing at prefill scale (1.3B shapes, 16384 tokens): two hot
    experts take 30 % of the assignments each and the null 15 % (the
    long-context decode workload's mix), stressing grouped-GEMM imbalance."""
    L = gen.make_layer("1p3b_bf16_prefill")
    N, E = 16384, L["cfg"]["E"]
    t = gen.expert_targets(dict(E=E, experts="skewed"))
    counts = np.floor(t * 2 * N).astype(np.int64)
    counts[3] += 2 * N - counts.sum()
    eidx, egate = _routing_with_counts(counts, 0, N, 2, 37)
    cm = _moe_case(L, N, eidx, egate, "skewed 30/30/15")
    note("hot expert rows", float(cm["exp_cnt"][1]))
