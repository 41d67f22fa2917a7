"""End-to-end parity of the composite layer calls against the CPU oracle.

The GPU runs every workload at full size, launched as the benchmark launches
it.  The comparison follows the protocol that makes every result well defined
(paper Sec. 3.2 (C) quantizer, Sec. 3.8 hard decisions):

1. routing decisions: bit exact for every token;
2. q, k, v (the GPU's stored projections): within the tolerance of the
   oracle's own projections;
3. the GPU's cache: codes, fp16 scale/zero and positions bit exact against
   the oracle's quantizer applied to the K/V tensor the GPU appended (its
   own k, v), every token of every compared sequence; a decode workload's
   whole pre-existing context bit exact against the oracle's quantizer of
   the generator's context (identical inputs);
4. discretely forced continuous outputs: the oracle attends over the cache
   its own quantizer builds from that k, v (so both sides read the same
   codes: a bf16 K that legitimately differs from the oracle's in its last
   bit can move a code by a whole quantization step) and recomputes o and x~
   in fp64 from the original inputs; its expert block takes the GPU's x~
   (just verified within tolerance: both sides hold x~ in bf16 and may round
   an element differently) and recomputes n2, the experts and x_out.  o, x~
   and x_out are held to the stated tolerance;
5. unforced: the GPU's x_out against the fully independent oracle, within
   1 + 2 x the spread that bf16 storage of the inter-operator tensors alone
   causes (measured on the CPU by test_activation_rounding_spread).

Every max err/bound is recorded and printed in the terminal summary."""
import numpy as np
import pytest
import torch

import gen
import oracle
import paper_2607_06601_amd as tr
from paper_2607_06601_amd.device import DeviceLayer, to_dev

from _common import ROUNDING_SPREAD, assert_close, layer, note, npy

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _taps(cfg, N, act_t):
    H, Hkv, dh, k, d = cfg["H"], cfg["Hkv"], cfg["dh"], cfg["k"], cfg["d"]
    t = dict(
        mode=torch.empty(N, H, dtype=torch.uint8, device=DEV),
        bit=torch.empty(N, dtype=torch.uint8, device=DEV),
        eidx=torch.empty(N, k, dtype=torch.int32, device=DEV),
        egate=torch.empty(N, k, dtype=torch.float32, device=DEV),
        o=torch.empty(N, H * dh, dtype=act_t, device=DEV),
        xt=torch.empty(N, d, dtype=act_t, device=DEV),
        q=torch.empty(N, H * dh, dtype=act_t, device=DEV),
        k=torch.empty(N, Hkv * dh, dtype=act_t, device=DEV),
        v=torch.empty(N, Hkv * dh, dtype=act_t, device=DEV))
    s = tr.Taps(mode=t["mode"].data_ptr(), bit=t["bit"].data_ptr(), eidx=t["eidx"].data_ptr(),
                egate=t["egate"].data_ptr(), o=t["o"].data_ptr(), xt=t["xt"].data_ptr(),
                q=t["q"].data_ptr(), k=t["k"].data_ptr(), v=t["v"].data_ptr())
    return t, s


def export_pool(c, cache, s, bi, n, act, Hkv, dh, G):
    tdt = torch.bfloat16 if act == "bf16" else torch.float32
    dt = torch.uint8 if bi < 3 else tdt
    ko = torch.zeros(n, Hkv, dh, dtype=dt, device=DEV)
    vo = torch.zeros_like(ko)
    ks = torch.zeros(n, Hkv, dh // G, 2, dtype=torch.int16, device=DEV)
    vs = torch.zeros_like(ks)
    pos = torch.zeros(n, dtype=torch.int32, device=DEV)
    tr.kv_export(c, cache, s, bi, 0, n, ko, vo, ks, vs, pos)
    torch.cuda.synchronize()
    return npy(ko), npy(vo), npy(ks), npy(vs), npy(pos)


def _f16_bits(a):
    return np.asarray(a).astype(np.int16).view(np.uint16)


def check_pool(c, cache, cfg, s, bi, ent, positions, first=0):
    """The slots [first, first + n) of pool (s, bi) hold, bit for bit, the
    oracle's quantization `ent` (store_kv's entry for that width) of the
    tokens at `positions`."""
    Hkv, dh, G, act = cfg["Hkv"], cfg["dh"], cfg["G"], cfg["act"]
    n = len(ent["tokens"])
    ko, vo, ks, vs, pos = export_pool(c, cache, s, bi, first + n, act, Hkv, dh, G)
    sl = slice(first, first + n)
    np.testing.assert_array_equal(pos[sl], positions)
    if bi == 3:
        np.testing.assert_array_equal(ko[sl].astype(np.float32), np.asarray(ent["kc"], np.float32))
        np.testing.assert_array_equal(vo[sl].astype(np.float32), np.asarray(ent["vc"], np.float32))
        return
    np.testing.assert_array_equal(ko[sl], ent["kc"])
    np.testing.assert_array_equal(vo[sl], ent["vc"])
    np.testing.assert_array_equal(_f16_bits(ks[sl][..., 0]), ent["ks"].view(np.uint16))
    np.testing.assert_array_equal(_f16_bits(ks[sl][..., 1]), ent["kz"].view(np.uint16))
    np.testing.assert_array_equal(_f16_bits(vs[sl][..., 0]), ent["vs"].view(np.uint16))
    np.testing.assert_array_equal(_f16_bits(vs[sl][..., 1]), ent["vz"].view(np.uint16))


def _codes_differ(own, forced):
    """Fraction of (token, kv head) cache entries whose codes or scale/zero
    differ between the oracle's quantization of its own K/V and of the GPU's."""
    tot = dif = 0
    for bi, a in own.items():
        if bi == 3:
            continue
        b = forced[bi]
        d = (a["kc"] != b["kc"]).any(-1) | (a["vc"] != b["vc"]).any(-1)
        for key in ("ks", "kz", "vs", "vz"):
            d |= (a[key].view(np.uint16) != b[key].view(np.uint16)).any(-1)
        dif += int(d.sum())
        tot += d.size
    return dif / max(tot, 1)


def _check_decisions(t, r):
    np.testing.assert_array_equal(npy(t["mode"]), r["mode"])
    np.testing.assert_array_equal(npy(t["bit"]), r["bit"])
    np.testing.assert_array_equal(npy(t["eidx"]), r["eidx"])
    np.testing.assert_allclose(npy(t["egate"]), r["egate"], rtol=2e-5, atol=1e-6)


def run_prefill(L, D=None):
    cfg = L["cfg"]
    D = D or DeviceLayer(L)
    c = D.cfg
    B, T = cfg["B"], cfg["T"]
    N = B * T
    cache = tr.KVCache(c, B, T)
    xo = torch.empty(N, cfg["d"], dtype=D.act, device=DEV)
    t, s = _taps(cfg, N, D.act)
    ws = tr.workspace(c, tr.OP_LAYER_PREFILL, B, T)
    tr.layer_prefill(c, B, T, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo, ws, taps=s)
    torch.cuda.synchronize()
    assert cache.status() == 0
    return xo, t, cache, c


# (workload, seed, sequences compared whole: None = all, variant); "dense" =
# the dense special case (every head full, every token 16-bit, one expert,
# k = 1) through the same kernels
PREFILL_CASES = [("tiny_f32_prefill", 0, None, None), ("160m_bf16_prefill", 1, None, None),
                 ("1p3b_bf16_prefill", 104, "first_last", None),
                 ("1p3b_bf16_prefill", 104, "first_last", "dense"),
                 ("160m_bf16_prefill", 1, "first_last", "per_token")]


def _variant(L, variant):
    """dense: the dense special case; per_token / per_group: one attention
    decision per token / per kv-head group (the granularity variants)."""
    if variant == "dense":
        return gen.dense_variant(L)
    if variant == "per_token":
        return gen.granularity_variant(L, 1)
    if variant == "per_group":
        return gen.granularity_variant(L, L["cfg"]["Hkv"])
    return L


@pytest.mark.parametrize("name,seed,which,variant", PREFILL_CASES)
def test_layer_prefill(name, seed, which, variant):
    L = _variant(layer(name, seed), variant)
    cfg = L["cfg"]
    act, B, T, H, Hkv, dh = (cfg[x] for x in ("act", "B", "T", "H", "Hkv", "dh"))
    xo, t, cache, c = run_prefill(L)
    seqs = list(range(B)) if which is None else sorted({0, B - 1})
    rows = np.concatenate([np.arange(b * T, (b + 1) * T) for b in seqs])
    # 1-2: decisions for every token, projections of the compared sequences;
    # the independent oracle's expert block on a sample of rows (step 5)
    sample = rows if which is None else np.unique(np.concatenate(
        [rows[:128], rows[-128:], gen.stream(seed, "rows").choice(rows, 256, replace=False)]))
    r0 = oracle.layer_prefill(L, sample)
    _check_decisions(t, r0)
    if variant == "dense":
        assert (r0["mode"] == oracle.MODE_FULL).all() and (r0["bit"] == 3).all()
        assert (r0["eidx"] == 1).all()
    gq, gk, gv = npy(t["q"]), npy(t["k"]), npy(t["v"])
    kv_in = {}
    for b in seqs:
        sl = slice(b * T, (b + 1) * T)
        assert_close(gq[sl], r0["q"][b].reshape(T, -1), act, "q")
        assert_close(gk[sl], r0["k"][b].reshape(T, -1), act, "k")
        assert_close(gv[sl], r0["v"][b].reshape(T, -1), act, "v")
        kv_in[b] = (gk[sl].reshape(T, Hkv, dh), gv[sl].reshape(T, Hkv, dh))
    # 3-4: the forced chain over every row of the compared sequences
    gxt = npy(t["xt"])
    r1 = oracle.layer_prefill(L, rows, kv_in=kv_in, o_in=npy(t["o"])[rows], xt_in=gxt[rows])
    flips = []
    for b in seqs:
        for bi, ent in r1["stored"][b].items():
            check_pool(c, cache, cfg, b, bi, ent, ent["tokens"])
        flips.append(_codes_differ(r0["stored"][b], r1["stored"][b]))
    note("cache entries moved by a last-bit K/V difference (fraction)", float(np.mean(flips)))
    assert np.mean(flips) < 1e-2
    assert_close(npy(t["o"])[rows], r1["o"].reshape(len(rows), -1), act, "o (forced codes)")
    assert_close(gxt[rows], r1["xt"], act, "x~ (forced o)")
    assert_close(npy(xo)[rows], r1["xout"], act, "x_out (forced x~)")
    # 5: unforced
    f = 1.0 + 2.0 * ROUNDING_SPREAD[name if variant is None else f"{name}/{variant}"]
    assert_close(npy(xo)[sample], r0["xout"], act, "x_out (unforced)", factor=f)


def test_layer_prefill_deterministic():
    L = layer("160m_bf16_prefill", 2)
    D = DeviceLayer(L)
    a = run_prefill(L, D)[0]
    b = run_prefill(L, D)[0]
    assert torch.equal(a, b)


def test_skip_and_null_tokens_keep_the_residual_on_device():
    L = layer("tiny_f32_prefill", 0)
    H, E = L["cfg"]["H"], L["cfg"]["E"]
    L["ca"] = np.tile(np.array([50.0, -50.0, -50.0], np.float32), H)
    L["ce"] = np.array([50.0] + [-50.0] * E, np.float32)
    xo, t, _, _ = run_prefill(L)
    assert (npy(t["mode"]) == 0).all() and (npy(t["eidx"]) == 0).all()
    np.testing.assert_array_equal(npy(t["xt"]), L["x"])
    np.testing.assert_array_equal(npy(xo), L["x"])


def fill_context(c, cache, cfg, act_t):
    """The decode workload's pre-existing context, appended one whole
    sequence per call (the benchmark's fill)."""
    ctx = cfg["ctx"]
    ws = tr.workspace(c, tr.OP_KV_APPEND, 1, ctx)
    for s in range(cfg["B"]):
        k, v = gen.context_kv(cfg, s)
        bits = gen.context_bits(cfg, s)
        tr.kv_append(c, cache, 1, ctx, to_dev(k.reshape(ctx, -1), act_t),
                     to_dev(v.reshape(ctx, -1), act_t), to_dev(bits, torch.uint8), ws,
                     seq_ids=torch.tensor([s], dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()


@pytest.mark.parametrize("name,nseq,variant", [("410m_bf16_decode", 12, None),
                                               ("1p3b_bf16_decode", 4, None),
                                               ("1p3b_bf16_decode", 2, "dense"),
                                               ("410m_bf16_decode", 6, "per_group")])
def test_layer_decode(name, nseq, variant):
    L = _variant(layer(name), variant)
    cfg = L["cfg"]
    D = DeviceLayer(L)
    c = D.cfg
    act, B, ctx, Hkv, dh = (cfg[x] for x in ("act", "B", "ctx", "Hkv", "dh"))
    cache = tr.KVCache(c, B, ctx + 16)
    fill_context(c, cache, cfg, D.act)
    assert cache.status() == 0
    xo = torch.empty(B, cfg["d"], dtype=D.act, device=DEV)
    t, s = _taps(cfg, B, D.act)
    tr.layer_decode(c, B, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo,
                    tr.workspace(c, tr.OP_LAYER_DECODE, B, 1), taps=s)
    torch.cuda.synchronize()
    assert cache.status() == 0
    np.testing.assert_array_equal(npy(cache.seq_len()), ctx + 1)
    seqs = np.unique(np.concatenate(
        [[0, B - 1], gen.stream(cfg["seed"], "seqs").choice(B, nseq, replace=False)]))
    seqs = [int(x) for x in seqs]
    r0 = oracle.layer_decode(L, seqs)
    _check_decisions(t, r0)
    if variant == "dense":
        assert (r0["mode"] == oracle.MODE_FULL).all() and (r0["bit"] == 3).all()
        assert (r0["eidx"] == 1).all()
    gq, gk, gv = npy(t["q"])[seqs], npy(t["k"])[seqs], npy(t["v"])[seqs]
    assert_close(gq, r0["q"].reshape(len(seqs), -1), act, "q")
    assert_close(gk, r0["k"].reshape(len(seqs), -1), act, "k")
    assert_close(gv, r0["v"].reshape(len(seqs), -1), act, "v")
    kv_in = {s_: (gk[i].reshape(1, Hkv, dh), gv[i].reshape(1, Hkv, dh))
             for i, s_ in enumerate(seqs)}
    gxt = npy(t["xt"])[seqs]
    r1 = oracle.layer_decode(L, seqs, kv_in=kv_in, o_in=npy(t["o"])[seqs], xt_in=gxt)
    bits_new = npy(t["bit"])
    for s_ in seqs:
        # the whole context fill, then the step's own token at the end of its pool
        _, _, stored, bits = oracle.decode_cache_seq(cfg, s_)
        for bi, ent in stored.items():
            check_pool(c, cache, cfg, s_, bi, ent, ent["tokens"])
        bi = int(bits_new[s_])
        first = int((bits == bi).sum())
        check_pool(c, cache, cfg, s_, bi, r1["stored"][s_][bi], [ctx], first=first)
    note("new tokens whose cache entry a last-bit K/V difference moved (fraction)",
         float(np.mean([_codes_differ(r0["stored"][s_], r1["stored"][s_]) for s_ in seqs])))
    assert_close(npy(t["o"])[seqs], r1["o"].reshape(len(seqs), -1), act, "o (forced codes)")
    assert_close(gxt, r1["xt"], act, "x~ (forced o)")
    assert_close(npy(xo)[seqs], r1["xout"], act, "x_out (forced x~)")
    f = 1.0 + 2.0 * ROUNDING_SPREAD[name if variant is None else f"{name}/{variant}"]
    assert_close(npy(xo)[seqs], r0["xout"], act, "x_out (unforced)", factor=f)


def test_layer_decode_wide_batch_rows_repeat():
    """320 decode rows: the 64 sequences of the 410M workload five times over
    (row b + 64 j holds row b's inputs and its own copy of b's context), so
    the step routes 640 expert assignments (the decode compaction's one-block
    scatter runs several rounds), appends 320 rows in one launch and takes
    the tile form of the router tail.  Every copy of a row must give the
    bit-identical result; against the 64-row step (one-block router tail)
    the decisions, q, the attention output and x~ are bit-identical, and
    x_out may differ only where the two tails' fp32 gates round a bf16
    element differently (one bf16 step)."""
    L = layer("410m_bf16_decode")
    cfg = L["cfg"]
    D = DeviceLayer(L)
    c = D.cfg
    B, ctx, R = cfg["B"], cfg["ctx"], 5
    BW = B * R
    runs = {}
    for nb in (B, BW):
        cache = tr.KVCache(c, nb, ctx + 16)
        ws = tr.workspace(c, tr.OP_KV_APPEND, 1, ctx)
        for s in range(B):
            k, v = gen.context_kv(cfg, s)
            bits = to_dev(gen.context_bits(cfg, s), torch.uint8)
            kd, vd = to_dev(k.reshape(ctx, -1), D.act), to_dev(v.reshape(ctx, -1), D.act)
            for j in range(nb // B):
                tr.kv_append(c, cache, 1, ctx, kd, vd, bits, ws,
                             seq_ids=torch.tensor([s + B * j], dtype=torch.int32, device=DEV))
        torch.cuda.synchronize()
        assert cache.status() == 0
        x = D.x.repeat(nb // B, 1)
        psi = D.psi.repeat(nb // B, 1)
        xo = torch.empty(nb, cfg["d"], dtype=D.act, device=DEV)
        t, s_ = _taps(cfg, nb, D.act)
        print(f"decode step of {nb} rows ({nb * cfg['k']} expert assignments)", flush=True)
        tr.layer_decode(c, nb, x, psi, D.rw, D.dw, D.mw, cache, xo,
                        tr.workspace(c, tr.OP_LAYER_DECODE, nb, 1), taps=s_)
        torch.cuda.synchronize()
        assert cache.status() == 0
        t["xout"] = xo
        runs[nb] = t
        del cache
    w, n = runs[BW], runs[B]
    for key in ("mode", "bit", "eidx", "egate", "q", "o", "xt", "xout"):
        for j in range(1, R):
            assert torch.equal(w[key][B * j:B * (j + 1)], w[key][:B]), (key, j)
    for key in ("mode", "bit", "eidx", "q", "o", "xt"):
        assert torch.equal(w[key][:B], n[key]), key
    ga, gb = w["egate"][:B].double(), n["egate"].double()
    note("wide decode: max rel gate difference against the 64-row step",
         float(((ga - gb).abs() / gb.abs().clamp_min(1e-30)).max()))
    assert torch.allclose(ga, gb, rtol=1e-5, atol=0)
    xa, xb = w["xout"][:B].double(), n["xout"].double()
    diff = (xa - xb).abs()
    note("wide decode: x_out elements differing from the 64-row step (fraction)",
         float((diff > 0).double().mean()))
    assert bool((diff <= 2.0 ** -7 * torch.maximum(xa.abs(), xb.abs())).all())
