"""Benchmark of the TriRoute routed-layer forward on one MI355X.

A step is one full routed-layer prefill (router, compaction, QKV + RoPE,
KV quantize/append, attention, O-proj, second norm, expert grouped GEMM,
combine) of the 1.3B-class workload, the largest that the benchmark's
configurations define: batch 4 x 4096 tokens, d 2048, 16 x 128 heads (4 kv
heads), window 512, 16 SwiGLU experts (d_ff 5632) + null, top-2, KV group 64,
bf16, seeded synthetic inputs and random-init weights.  Inputs are resident in
HBM before timing; every step writes a fresh cache; L2 and the 256 MB
Infinity Cache are flushed before each timed step by reading a 1 GiB buffer
(a read, so that no dirty lines are left whose write-back would land in the
timed region).  Each step is bracketed by HIP events on the launch stream.

Also reported, as extra keys of the one JSON line:
  roofline      the MoE sublayer (triroute_moe) of the headline workload:
                achieved bf16 MFMA rate of the algorithmic expert FLOPs
  prefill_160m  the 160M-class prefill (8 x 2048) on seeds 1, 2, 3 and their
                median, with its MoE sublayer
  decode_410m / decode_1p3b
                the decode steps (64 x 8192 and 32 x 32768 context) with the
                decode attention's achieved HBM bandwidth; the same attention
                with every head in full mode over the routed mixed-width cache
                (bandwidth stress point); and the dense special case (all
                heads full, every token 16-bit, one expert, k = 1) through the
                same kernels, with routed / dense tokens/s and the cost-model
                fractions of the routed step
  dense_1p3b_prefill
                the dense special case of the headline workload
  cpu_baseline  the CPU oracle on a bounded sample of the headline workload
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2516.6  # MI355X dense bf16 MFMA, TFLOP/s (256 CU x 2.4 GHz x 4096)

HEADLINE = "1p3b_bf16_prefill"
SMALL = "160m_bf16_prefill"
DECODES = {"decode_410m": "410m_bf16_decode", "decode_1p3b": "1p3b_bf16_decode"}
METRIC = "routed-layer tokens/s (prefill, decode); decode-attn HBM GB/s; MoE MFMA util"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extra", action="store_true",
                   help="the headline workload only (no 160M, decode or dense legs)")
    p.add_argument("--only", default=None,
                   choices=("prefill_1p3b", "prefill_160m", "moe_1p3b", "moe_160m",
                            "decode_410m", "decode_1p3b", "attn_410m", "attn_1p3b",
                            "stack_410m", "relaxed_1p3b"),
                   help="profile one leg alone (prints its section only); moe_* time the "
                        "MoE sublayer, attn_* the decode attention, and both then run a "
                        "256 MiB copy for counter calibration")
    p.add_argument("--summarize-pmc", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "KERNEL_REGEX"),
                   default=None,
                   help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; csv output) "
                        "into per-launch HBM bytes of the kernels matching KERNEL_REGEX, "
                        "scaled by the 256 MiB copy in the same runs")
    return p.parse_args()


class CacheFlush:
    """Evicts L2 and the Infinity Cache by reading a 1 GiB buffer."""

    def __init__(self, torch, dev):
        # fp32, so that the reduction reads the buffer as it is (no widening copy)
        self.buf = torch.ones(1 << 28, dtype=torch.float32, device=dev)

    def __call__(self):
        self.buf.sum()


class Ctx:
    """Modules and shared objects of one benchmark run."""

    def __init__(self, args):
        import numpy as np
        import torch

        import gen
        import paper_2607_06601_amd as tr
        from paper_2607_06601_amd.device import DeviceLayer, to_dev
        self.args, self.np, self.torch, self.gen, self.tr = args, np, torch, gen, tr
        self.DeviceLayer, self.to_dev = DeviceLayer, to_dev
        self.dev = "cuda"
        self.flush = CacheFlush(torch, self.dev)
        self._layer = (None, None)

    def layer(self, name, seed=None):
        """The generator's layer (the last one is kept: the headline, its
        dense case and the CPU baseline share it; callers copy before they
        change anything)."""
        key = (name, seed)
        if self._layer[0] != key:
            self._layer = (None, None)
            self._layer = (key, self.gen.make_layer(name, seed))
        return self._layer[1]

    def timed(self, fn, steps, before=None):
        """Mean and per-step ms of `steps` calls of fn(i), each preceded by a
        cache flush, bracketed by HIP events on the current stream."""
        torch = self.torch
        stream = torch.cuda.current_stream()
        ev = []
        torch.cuda.synchronize()
        for i in range(steps):
            if before:
                before(i)
            self.flush()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn(i)
            e1.record(stream)
            ev.append((e0, e1))
        torch.cuda.synchronize()
        ms = [a.elapsed_time(b) for a, b in ev]
        return float(self.np.mean(ms)), ms


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): the routed layer is "
              "measured on a single MI355X",
              file=sys.stderr)
        sys.exit(2)
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc)
        return
    import torch
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    cx = Ctx(args)
    cx.tr.lib()
    if args.only:
        leg = args.only
        if leg in ("prefill_1p3b", "moe_1p3b"):
            r = bench_prefill(cx, HEADLINE, None, args.steps, args.warmup, moe_only=leg == "moe_1p3b")
        elif leg in ("prefill_160m", "moe_160m"):
            r = bench_prefill(cx, SMALL, 1, args.steps, args.warmup, moe_only=leg == "moe_160m")
        elif leg == "stack_410m":
            r = bench_stack(cx, args.steps, args.warmup, None)
        elif leg == "relaxed_1p3b":
            r = bench_relaxed(cx, args.steps, args.warmup)
        else:
            name = DECODES["decode_410m" if leg.endswith("410m") else "decode_1p3b"]
            r = bench_decode(cx, name, args.steps, args.warmup, attn_only=leg.startswith("attn"))
        if leg.startswith(("moe", "attn")):
            copy_calibration(torch)
        print(json.dumps({leg: r}), flush=True)
        return

    K, W = args.steps, args.warmup
    head = bench_prefill(cx, HEADLINE, None, K, W)
    N = head["B"] * head["T"]
    cfg = cx.gen.CONFIGS[HEADLINE]
    out = {
        "metric": METRIC,
        "value": round(N / (head["ms"] * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(head["ms"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded generator, random-init weights)",
        "config": {"workload": "1.3B-class TriRoute " + describe(cfg),
                   "global_batch": head["B"], "seq_len": head["T"],
                   "parallelism": "single GPU"},
        "roofline": head["roofline"],
        "timing": {"per_step_ms_min": round(min(head["step_ms"]), 4),
                   "per_step_ms_max": round(max(head["step_ms"]), 4),
                   "cache_flush_per_step": "1 GiB read"},
    }
    if not args.no_extra:
        ks, ws = min(K, 10), min(W, 3)
        out["prefill_160m"] = bench_small_seeds(cx, ks, ws)
        for key, name in DECODES.items():
            out[key] = bench_decode(cx, name, ks, ws)
        out["stack_410m_decode"] = bench_stack(cx, ks, ws, out["decode_410m"]["ms_per_step"])
        out["dense_1p3b_prefill"] = bench_dense_prefill(cx, ks, ws, head)
        out["granularity_1p3b_prefill"] = bench_granularity(cx, ks, ws, head)
        out["relaxed_1p3b_router"] = bench_relaxed(cx, ks, ws)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cx.layer(HEADLINE))
    print(json.dumps(out), flush=True)


def describe(cfg):
    """The workload's sizes in words."""
    if cfg["kind"] == "prefill":
        head = f"layer prefill: batch {cfg['B']} x seq {cfg['T']}"
    else:
        head = (f"decode step: {cfg['B']} sequences x 1 new token, context {cfg['ctx']} (bits "
                + "/".join(f"{round(100 * f)}" for f in cfg["ctx_bits"]) + " % for 2/4/8/16)")
    ex = {"skewed": "skewed", "uniform": "uniform"}.get(cfg["experts"], cfg["experts"])
    return (f"{head}, d {cfg['d']}, {cfg['H']}x{cfg['dh']} heads ({cfg['Hkv']} kv), window "
            f"{cfg['w']}, {cfg['E']} SwiGLU experts d_ff {cfg['d_ff']} + null, top-{cfg['k']} "
            f"({ex} routing), KV group {cfg['G']}, {cfg['act']}")


def bench_prefill(cx, name, seed, steps, warmup, moe_only=False, L=None):
    """Timed triroute_layer_prefill steps of one prefill workload, then its
    MoE sublayer alone on the same routed inputs."""
    np, torch, tr = cx.np, cx.torch, cx.tr
    if L is None:
        L = cx.layer(name, seed)
    cfg = L["cfg"]
    B, T, d, k = (cfg[x] for x in ("B", "T", "d", "k"))
    N = B * T
    D = cx.DeviceLayer(L)
    c = D.cfg
    ws = tr.workspace(c, tr.OP_LAYER_PREFILL, B, T)
    xo = torch.empty(N, d, dtype=D.act, device=cx.dev)
    eidx_t = torch.empty(N, k, dtype=torch.int32, device=cx.dev)
    egate_t = torch.empty(N, k, dtype=torch.float32, device=cx.dev)
    xt_t = torch.empty(N, d, dtype=D.act, device=cx.dev)
    taps = tr.Taps(eidx=eidx_t.data_ptr(), egate=egate_t.data_ptr(), xt=xt_t.data_ptr())
    warm = tr.KVCache(c, B, T)
    for _ in range(max(warmup, 1)):
        for s in range(B):
            warm.reset_seq(s)
        tr.layer_prefill(c, B, T, D.x, D.psi, D.rw, D.dw, D.mw, warm, xo, ws, taps=taps)
    torch.cuda.synchronize()
    res = {"B": B, "T": T}
    if not moe_only:
        caches = [tr.KVCache(c, B, T) for _ in range(steps)]
        ms, step_ms = cx.timed(lambda i: tr.layer_prefill(c, B, T, D.x, D.psi, D.rw, D.dw, D.mw,
                                                           caches[i], xo, ws, taps=taps), steps)
        for cc in caches:
            assert cc.status() == 0
        del caches
        res.update(ms=ms, step_ms=step_ms, tokens_per_s=round(N / (ms * 1e-3), 1))
    del warm
    res["roofline"] = bench_moe(cx, D, c, B, T, eidx_t, egate_t, xt_t, xo, name, steps)
    return res


def bench_moe(cx, D, c, B, T, eidx_t, egate_t, xt_t, xo, name, steps):
    """The MoE sublayer (triroute_moe: rmsnorm2, grouped GEMM gate/up +
    SwiGLU, grouped GEMM down, combine) alone on the routed inputs of the last
    prefill step: achieved bf16 MFMA rate of the algorithmic expert FLOPs
    (6 d d_ff per real assignment; norm and combine time included)."""
    np, torch, tr = cx.np, cx.torch, cx.tr
    d, dff = c.d_model, c.d_ff
    N = B * T
    n_real = int((eidx_t.cpu().numpy() != 0).sum())
    moe_flops = 6.0 * d * dff * n_real
    cmp = tr.CompactionBuffers(c, B, T)
    n1 = torch.empty(N, d, dtype=D.act, device=cx.dev)
    mode = torch.empty(N, c.n_heads, dtype=torch.uint8, device=cx.dev)
    bit = torch.empty(N, dtype=torch.uint8, device=cx.dev)
    tr.router(c, B, T, D.x, D.psi, D.rw, n1, mode, bit, eidx_t, egate_t, cmp.struct,
              tr.workspace(c, tr.OP_ROUTER, B, T))
    moe_ws = tr.workspace(c, tr.OP_MOE, N, 1)
    for _ in range(3):
        tr.moe(c, N, xt_t, D.dw, D.mw, eidx_t, egate_t, cmp.struct, xo, moe_ws)
    ms, _ = cx.timed(lambda i: tr.moe(c, N, xt_t, D.dw, D.mw, eidx_t, egate_t, cmp.struct, xo,
                                      moe_ws), steps)
    tflops = moe_flops / (ms * 1e-3) / 1e12
    prof = {HEADLINE: "moe_1p3b_prefill_traffic.txt", SMALL: "moe_160m_prefill_traffic.txt"}
    return {"kernel": "triroute_moe (rmsnorm2, grouped GEMM gate/up + SwiGLU, grouped GEMM "
                      "down, combine)",
            "bound": "mfma", "achieved": round(tflops, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": stored_traffic(prof.get(name), MOE_SOURCES),
            "algorithmic": f"6*d*d_ff FLOP x {n_real} real assignments = "
                           f"{moe_flops / 1e9:.1f} GFLOP per launch",
            "avg_ms": round(ms, 4)}


def bench_small_seeds(cx, steps, warmup):
    """The 160M-class prefill on its three seeds; the median is the figure."""
    per = {}
    moe = None
    for seed in cx.gen.CONFIGS[SMALL]["seeds"]:
        r = bench_prefill(cx, SMALL, seed, steps, warmup)
        per[str(seed)] = {"tokens_per_s": r["tokens_per_s"], "ms_per_step": round(r["ms"], 4),
                          "moe_frac": r["roofline"]["frac"]}
        if moe is None:
            moe = r["roofline"]
    tps = [v["tokens_per_s"] for v in per.values()]
    return {"workload": "160M-class " + describe(cx.gen.CONFIGS[SMALL]),
            "tokens_per_s_median": round(statistics.median(tps), 1), "seeds": per,
            "steps": steps, "moe_seed1": moe}


def source_digest(*names):
    """sha256 over kernel sources (package csrc/), to tell whether stored
    counter readings still describe the kernels as built."""
    import hashlib
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2607_06601_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


MOE_SOURCES = ("gemm_mfma.hip", "misc.hip", "common.hpp", "kernels.hpp", "api.cpp")
DECODE_ATTN_SOURCES = ("attn_mfma.hip", "common.hpp", "kernels.hpp", "api.cpp")


def stored_traffic(name, sources):
    """HBM bytes per launch from a committed counter summary under profiles/
    (FETCH_SIZE + WRITE_SIZE, scaled by the plain-copy calibration), or None
    when it is missing or was taken from other kernel sources."""
    if not name:
        return None
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_digest") != source_digest(*sources):
        return None
    try:
        return int(float(kv["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def copy_calibration(torch):
    """A plain device copy of 256 MiB: the reference reading for the FETCH_SIZE
    / WRITE_SIZE counters (kernel name contains 'copy' or 'elementwise')."""
    n = 256 << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    return n


def slot_bytes(cfg):
    """Packed K+V bytes of one cached token per kv head at each width,
    fp16 scale/zero included (16-bit: the bf16 values only)."""
    dh, G = cfg["dh"], cfg["G"]
    return [2 * dh * b / 8 + (2 * (dh // G) * 4 if b < 16 else 0) for b in (2, 4, 8, 16)]


def decode_attn_bytes(cfg, mode, bits_per_seq):
    """Algorithmic bytes the routed decode attention must read: per (sequence,
    kv head), the union of the key ranges its query heads need (full -> all
    P+1 keys, local -> last w, skip -> none) x packed K+V bytes incl. fp16
    scale/zero."""
    import numpy as np
    H, Hkv, w = cfg["H"], cfg["Hkv"], cfg["w"]
    grp = H // Hkv
    per_tok = np.array(slot_bytes(cfg))
    total = 0.0
    for s, bits in enumerate(bits_per_seq):
        P1 = len(bits)
        full_b = per_tok[bits].sum()
        loc_b = per_tok[bits[max(0, P1 - w):]].sum()
        for g in range(Hkv):
            m = mode[s, g * grp:(g + 1) * grp].max()
            total += full_b if m == 2 else loc_b if m == 1 else 0.0
    return total


def decode_cost(cfg, mode, bits_per_seq, eidx):
    """Cost-model terms of one decode step (paper Sec. 3.5 per-token costs,
    App. A): attention MACs 2 d_h per head and key (local: the window's w
    keys, full: all P + 1), KV memory 2 d_kv b bits per cached token, expert
    MACs 3 d d_f per real assignment (reading R27)."""
    import numpy as np
    H, dh, w, d, dff = cfg["H"], cfg["dh"], cfg["w"], cfg["d"], cfg["d_ff"]
    dkv = cfg["Hkv"] * dh
    attn = kv = 0.0
    for s, bits in enumerate(bits_per_seq):
        P1 = len(bits)
        for h in range(H):
            m = int(mode[s, h])
            attn += 2 * dh * (0 if m == 0 else min(P1, w) if m == 1 else P1)
        kv += 2 * dkv * float(np.sum(np.array([2, 4, 8, 16])[bits]))
    ffn = 3.0 * d * dff * float((eidx != 0).sum())
    return {"attn_macs": attn, "kv_bits": kv, "ffn_macs": ffn}


def fill_decode_cache(cx, c, cache, cfg, act_t, dense=False):
    """The workload's pre-existing context: the generator's K/V at its
    per-position widths (all 16-bit for the dense case)."""
    np, torch, tr, gen = cx.np, cx.torch, cx.tr, cx.gen
    ctx = cfg["ctx"]
    ws = tr.workspace(c, tr.OP_KV_APPEND, 1, ctx)
    bits_all = []
    for s in range(cfg["B"]):
        kk, vv = gen.context_kv(cfg, s)
        bits = np.full(ctx, 3, np.uint8) if dense else gen.context_bits(cfg, s)
        bits_all.append(bits)
        tr.kv_append(c, cache, 1, ctx, cx.to_dev(kk.reshape(ctx, -1), act_t),
                     cx.to_dev(vv.reshape(ctx, -1), act_t), cx.to_dev(bits, torch.uint8), ws,
                     seq_ids=torch.tensor([s], dtype=torch.int32, device=cx.dev))
    torch.cuda.synchronize()
    return bits_all


PAGE_TILES = 8


def decode_pages(cx, cfg, extra, slack=4):
    """Pages per width of a paged cache that holds the workload's context and
    `extra` more tokens a sequence."""
    per = PAGE_TILES * (4096 // cfg["dh"])
    need = [slack] * 4
    for s in range(cfg["B"]):
        cnt = cx.np.bincount(cx.gen.context_bits(cfg, s), minlength=4)
        for bi in range(4):
            need[bi] += -(-(int(cnt[bi]) + extra) // per)
    return need


def run_decode_steps(cx, L, steps, warmup, dense=False, paged=False):
    """Timed decode steps of one layer over a freshly filled cache (contiguous
    pools, or a paged cache); returns the step time, the step's decisions and
    the cache."""
    np, torch, tr = cx.np, cx.torch, cx.tr
    cfg = L["cfg"]
    B, d, H, k = cfg["B"], cfg["d"], cfg["H"], cfg["k"]
    D = cx.DeviceLayer(L)
    c = D.cfg
    cap = cfg["ctx"] + warmup + steps + 1
    pages = (PAGE_TILES, decode_pages(cx, cfg, warmup + steps + 1)) if paged else None
    cache = tr.KVCache(c, B, cap, pages=pages)
    bits_all = fill_decode_cache(cx, c, cache, cfg, D.act, dense)
    ws = tr.workspace(c, tr.OP_LAYER_DECODE, B, 1)
    xo = torch.empty(B, d, dtype=D.act, device=cx.dev)
    t = dict(mode=torch.empty(B, H, dtype=torch.uint8, device=cx.dev),
             bit=torch.empty(B, dtype=torch.uint8, device=cx.dev),
             eidx=torch.empty(B, k, dtype=torch.int32, device=cx.dev),
             q=torch.empty(B, H * cfg["dh"], dtype=D.act, device=cx.dev))
    taps = tr.Taps(**{n: x.data_ptr() for n, x in t.items()})
    for _ in range(warmup):
        tr.layer_decode(c, B, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo, ws, taps=taps)
    ms, _ = cx.timed(lambda i: tr.layer_decode(c, B, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo, ws,
                                               taps=taps), steps)
    assert cache.status() == 0
    seq_len = cache.seq_len().cpu().numpy()
    extra = t["bit"].cpu().numpy()
    ctx = cfg["ctx"]
    bits_now = [np.concatenate([bits_all[s], np.full(seq_len[s] - ctx, extra[s], np.uint8)])
                for s in range(B)]
    return dict(ms=ms, D=D, c=c, cache=cache, t=t, bits=bits_now,
                eidx=t["eidx"].cpu().numpy())


STACK_LAYERS = 8


def bench_stack(cx, steps, warmup, single_ms):
    """One decode step through a stack of STACK_LAYERS routed layers of the
    410M-class decode workload (triroute_stack_decode: the next layer's side
    features from the previous layer's decisions on the device), every layer
    over its own cache holding the workload's context (the same K/V values
    and widths in every layer)."""
    np, torch, tr = cx.np, cx.torch, cx.tr
    name = "410m_bf16_decode"
    Ls = cx.gen.make_stack(name, STACK_LAYERS)
    cfg = Ls[0]["cfg"]
    B, d = cfg["B"], cfg["d"]
    Ds = [cx.DeviceLayer(L) for L in Ls]
    c = Ds[0].cfg
    caches = [tr.KVCache(c, B, cfg["ctx"] + warmup + steps + 1) for _ in Ds]
    ctx = cfg["ctx"]
    aws = tr.workspace(c, tr.OP_KV_APPEND, 1, ctx)
    for sq in range(B):
        kk, vv = cx.gen.context_kv(cfg, sq)
        k_t = cx.to_dev(kk.reshape(ctx, -1), Ds[0].act)
        v_t = cx.to_dev(vv.reshape(ctx, -1), Ds[0].act)
        b_t = cx.to_dev(cx.gen.context_bits(cfg, sq), torch.uint8)
        sid = torch.tensor([sq], dtype=torch.int32, device=cx.dev)
        for cache in caches:
            tr.kv_append(c, cache, 1, ctx, k_t, v_t, b_t, aws, seq_ids=sid)
    torch.cuda.synchronize()
    ws = tr.workspace(c, tr.OP_STACK_DECODE, B, 1)
    xo = torch.empty(B, d, dtype=Ds[0].act, device=cx.dev)
    layers = [(D.rw, D.dw, D.mw) for D in Ds]
    run = lambda i: tr.stack_decode(c, B, Ds[0].x, Ds[0].psi, layers, caches, xo, ws)
    for _ in range(warmup):
        run(0)
    ms, _ = cx.timed(run, steps)
    assert all(ca.status() == 0 for ca in caches)
    return {"workload": f"{STACK_LAYERS}-layer stack of the 410M-class decode step (64 sequences, "
                        "context 8192 per layer), one decode step through every layer",
            "layers": STACK_LAYERS, "tokens_per_s": round(B / (ms * 1e-3), 1),
            "ms_per_step": round(ms, 4), "ms_per_layer": round(ms / STACK_LAYERS, 4),
            "single_layer_ms": None if single_ms is None else round(single_ms, 4)}


def bench_attn(cx, r, cfg, mode_t, steps, label):
    """The decode attention alone over the cache as it stands, with the
    given per-head modes: achieved HBM bandwidth of the algorithmic bytes."""
    tr, torch = cx.tr, cx.torch
    B, H = cfg["B"], cfg["H"]
    nbytes = decode_attn_bytes(cfg, mode_t.cpu().numpy(), r["bits"])
    o = torch.empty(B, H * cfg["dh"], dtype=r["D"].act, device=cx.dev)
    aws = tr.workspace(r["c"], tr.OP_ATTN_DECODE, B, 1)
    for _ in range(3):
        tr.attn_decode(r["c"], B, r["t"]["q"], r["cache"], mode_t, o, aws)
    ms, _ = cx.timed(lambda i: tr.attn_decode(r["c"], B, r["t"]["q"], r["cache"], mode_t, o,
                                              aws), steps)
    gbs = nbytes / (ms * 1e-3) / 1e9
    prof = {"410m_bf16_decode": "attn_decode_410m_traffic.txt",
            "1p3b_bf16_decode": "attn_decode_1p3b_traffic.txt"}
    return {"modes": label, "bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "algorithmic_bytes": int(nbytes),
            "avg_ms": round(ms, 4),
            "traffic": (stored_traffic(prof.get(cfg["name"]), DECODE_ATTN_SOURCES)
                        if label == "routed" else None)}


def bench_decode(cx, name, steps, warmup, attn_only=False):
    np, torch = cx.np, cx.torch
    L = cx.gen.make_layer(name)
    cfg = L["cfg"]
    B = cfg["B"]
    r = run_decode_steps(cx, L, steps, warmup)
    cls = "410M" if name.startswith("410m") else "1.3B"
    out = {"workload": f"{cls}-class " + describe(cfg),
           "tokens_per_s": round(B / (r["ms"] * 1e-3), 1), "ms_per_step": round(r["ms"], 4),
           "attn": bench_attn(cx, r, cfg, r["t"]["mode"], steps, "routed")}
    if attn_only:
        return out
    full = torch.full_like(r["t"]["mode"], 2)
    out["attn_all_full"] = bench_attn(cx, r, cfg, full, steps, "every head full (routed widths)")
    routed_cost = decode_cost(cfg, r["t"]["mode"].cpu().numpy(), r["bits"], r["eidx"])
    cont_mib = r["cache"].nbytes / 2 ** 20
    del r
    torch.cuda.empty_cache()
    # the same steps over a paged cache (pages of PAGE_TILES tiles per width)
    rp = run_decode_steps(cx, L, steps, warmup, paged=True)
    out["paged"] = {"page_tiles": PAGE_TILES,
                    "cache_mib": round(rp["cache"].nbytes / 2 ** 20, 1),
                    "contiguous_cache_mib": round(cont_mib, 1),
                    "tokens_per_s": round(B / (rp["ms"] * 1e-3), 1),
                    "ms_per_step": round(rp["ms"], 4),
                    "paged_over_contiguous_ms": round(rp["ms"] / out["ms_per_step"], 3)}
    del rp
    torch.cuda.empty_cache()
    # the dense special case through the same kernels
    Ld = cx.gen.dense_variant(L)
    del L
    rd = run_decode_steps(cx, Ld, steps, warmup, dense=True)
    dcfg = Ld["cfg"]
    assert (rd["t"]["mode"].cpu().numpy() == 2).all() and (rd["eidx"] == 1).all()
    dense_cost = decode_cost(dcfg, rd["t"]["mode"].cpu().numpy(), rd["bits"], rd["eidx"])
    out["dense"] = {
        "workload": "dense special case: every head full, every token 16-bit, one SwiGLU "
                    "expert (d_ff %d), k = 1" % dcfg["d_ff"],
        "tokens_per_s": round(B / (rd["ms"] * 1e-3), 1), "ms_per_step": round(rd["ms"], 4),
        "attn": bench_attn(cx, rd, dcfg, rd["t"]["mode"], steps, "dense: all full, 16-bit")}
    out["routed_over_dense_tokens_per_s"] = round(rd["ms"] / out["ms_per_step"], 3)
    out["cost_model_routed_over_dense"] = {
        key: round(routed_cost[key] / dense_cost[key], 4) for key in routed_cost}
    del rd
    torch.cuda.empty_cache()
    return out


def bench_dense_prefill(cx, steps, warmup, head):
    """The dense special case of the headline workload through the same
    kernels (NEXT to the routed headline figure)."""
    Ld = cx.gen.dense_variant(cx.layer(HEADLINE))
    r = bench_prefill(cx, HEADLINE, None, steps, warmup, L=Ld)
    N = r["B"] * r["T"]
    return {"workload": "dense special case of the 1.3B-class prefill: every head full, every "
                        "token 16-bit, one SwiGLU expert (d_ff 5632), k = 1",
            "tokens_per_s": round(N / (r["ms"] * 1e-3), 1), "ms_per_step": round(r["ms"], 4),
            "routed_over_dense_tokens_per_s": round(r["ms"] / head["ms"], 3)}


def bench_granularity(cx, steps, warmup, head):
    """The headline prefill with one attention decision per token and per
    kv-head group instead of per head (the granularity variants) through the
    same kernels."""
    base = cx.layer(HEADLINE)
    out = {}
    for label, groups in (("per_token", 1), ("per_kv_group", base["cfg"]["Hkv"])):
        L = cx.gen.granularity_variant(base, groups)
        r = bench_prefill(cx, HEADLINE, None, steps, warmup, L=L)
        N = r["B"] * r["T"]
        out[label] = {"attn_groups": groups, "tokens_per_s": round(N / (r["ms"] * 1e-3), 1),
                      "ms_per_step": round(r["ms"], 4),
                      "over_per_head_tokens_per_s": round(head["ms"] / r["ms"], 3)}
    return out


def bench_relaxed(cx, steps, warmup):
    """The training-time relaxed controller forward (whitening, ST-Gumbel,
    expected costs, losses, dual step, compaction) and its backward pass on
    the headline prefill's tokens, beside the inference controller
    (triroute_router) on the same tokens."""
    torch, tr, np = cx.torch, cx.tr, cx.np
    L = cx.layer(HEADLINE)
    cfg = L["cfg"]
    B, T, H, E, k = cfg["B"], cfg["T"], cfg["H"], cfg["E"], cfg["k"]
    N = B * T
    R = cx.gen.relax_inputs(L)
    D = cx.DeviceLayer(L, moe=False)
    c = D.cfg
    dev, f32 = cx.dev, torch.float32
    t = {n: cx.to_dev(R[n], f32) for n in ("g_attn", "g_bits", "white_mu", "white_sd")}
    t["pos"] = cx.to_dev(R["pos"], torch.int32)
    t["dual"] = cx.to_dev(np.asarray(R["dual"]), torch.float64)
    p = tr.RelaxParams(g_attn=t["g_attn"].data_ptr(), g_bits=t["g_bits"].data_ptr(),
                       pos=t["pos"].data_ptr(), white_mu=t["white_mu"].data_ptr(),
                       white_sd=t["white_sd"].data_ptr(), white_eps=R["white_eps"],
                       tau_a=R["tau_a"], tau_b=R["tau_b"], zeta=R["zeta"], alpha=R["alpha"],
                       beta=R["beta"], gamma=R["gamma"], dual=t["dual"].data_ptr(),
                       dual_lr=R["dual_lr"], dual_ema=R["dual_ema"])
    p.c_target[0], p.c_target[1] = R["c_target"]
    o = [torch.empty(N, H, 3, dtype=f32, device=dev), torch.empty(N, 4, dtype=f32, device=dev),
         torch.empty(N, dtype=f32, device=dev), torch.empty(N, dtype=f32, device=dev),
         torch.empty(tr.RELAX_NSTAT, dtype=torch.float64, device=dev)]
    out = tr.RelaxOut(*(x.data_ptr() for x in o), None, None, None, None, None)
    n1 = torch.empty(N, cfg["d"], dtype=D.act, device=dev)
    mode = torch.empty(N, H, dtype=torch.uint8, device=dev)
    bit = torch.empty(N, dtype=torch.uint8, device=dev)
    eidx = torch.empty(N, k, dtype=torch.int32, device=dev)
    egate = torch.empty(N, k, dtype=f32, device=dev)
    cmp = tr.CompactionBuffers(c, B, T)
    ws_r = tr.workspace(c, tr.OP_ROUTER_RELAXED, B, T)
    ws_i = tr.workspace(c, tr.OP_ROUTER, B, T)

    def relaxed(_):
        tr.router_relaxed(c, B, T, D.x, D.psi, D.rw, p, n1, mode, bit, eidx, egate, cmp.struct,
                          out, ws_r)

    def inference(_):
        tr.router(c, B, T, D.x, D.psi, D.rw, n1, mode, bit, eidx, egate, cmp.struct, ws_i)

    # the backward pass on the same tokens: upstream gradients of the soft
    # samples and gates drawn N(0, 1), balance factors stepped each call
    o.append(torch.empty(2, E + 1, dtype=torch.float64, device=dev))
    out.usage_exp = o[-1].data_ptr()
    A = H
    up = [cx.to_dev(cx.gen.normal(9, n, shp), f32) for n, shp in
          (("bwd_ga", (N, A, 3)), ("bwd_gb", (N, 4)), ("bwd_gg", (N, k)))]
    lam = cx.to_dev(np.asarray(R["dual"][:2]), torch.float64)
    rho = torch.ones(3, dtype=torch.float64, device=dev)
    gin = tr.RelaxGradIn(g_attn=up[0].data_ptr(), g_bits=up[1].data_ptr(), g_gate=up[2].data_ptr(),
                         lambda_=lam.data_ptr(), rho=rho.data_ptr(), rho_m=0.01)
    shapes = dict(dW1=(128, cfg["d"] + 8), db1=(128,), dW2=(128, 128), db2=(128,), dgr=(128,),
                  dWa=(3 * H, 128), dca=(3 * H,), dWe=(E + 1, 128), dce=(E + 1,), dWb=(4, 128),
                  dcb=(4,), dg1=(cfg["d"],), dx=(N, cfg["d"]), dpsi=(N, 8))
    gt = {n: torch.empty(shp, dtype=f32, device=dev) for n, shp in shapes.items()}
    gout = tr.RelaxGradOut(**{n: v.data_ptr() for n, v in gt.items()})
    ws_b = tr.workspace(c, tr.OP_ROUTER_RELAXED_BACKWARD, B, T)

    def backward(_):
        tr.router_relaxed_backward(c, B, T, D.x, D.psi, D.rw, p, out, eidx, egate, gin, gout, ws_b)

    for i in range(warmup):
        relaxed(i)
        inference(i)
    relaxed(0)
    for i in range(warmup):
        backward(i)
    ms_r, _ = cx.timed(relaxed, steps)
    ms_i, _ = cx.timed(inference, steps)
    relaxed(0)
    ms_b, _ = cx.timed(backward, steps)
    return {"workload": f"relaxed controller forward on the 1.3B-class prefill tokens ({B} x {T}): "
                        "per-axis whitening, ST-Gumbel (attention per head, bits), top-k experts, "
                        "expected costs, balance / z / entropy losses, dual step, compaction",
            "tokens_per_s": round(N / (ms_r * 1e-3), 1), "ms_per_call": round(ms_r, 4),
            "inference_router_ms": round(ms_i, 4),
            "relaxed_over_inference_ms": round(ms_r / ms_i, 3),
            "backward_ms_per_call": round(ms_b, 4),
            "backward_tokens_per_s": round(N / (ms_b * 1e-3), 1)}


def summarize_pmc(fetch_dir, write_dir, regex):
    """Per-launch HBM bytes of the kernels matching `regex` (one dispatch of
    each per launch) from two rocprofv3 counter runs, each counter scaled by
    what it reads for the 256 MiB copy of copy_calibration(), which reads and
    writes 256 MiB."""
    import csv
    import glob
    import re

    pat = re.compile(regex)

    def read(d, counter):
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(f) as fh:
                for r in csv.DictReader(fh):
                    if r.get("Counter_Name") == counter:
                        rows.append((r["Kernel_Name"], int(r.get("Dispatch_Id", 0)),
                                     float(r["Counter_Value"])))
        return rows

    out = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = read(d, counter)
        # the 256 MiB device copy (hipMemcpy D2D kernel) reads and writes 256 MiB
        copy = sorted(v for n, _, v in rows if "copyBuffer" in n and v > 0.25 * (256 << 10))
        ref = (256 << 10) / copy[len(copy) // 2] if copy else float("nan")
        per_kernel = {}
        for n, _, v in rows:
            if pat.search(n):
                per_kernel.setdefault(n, []).append(v)
        out[counter] = (ref, {n: sum(v) / len(v) for n, v in per_kernel.items()},
                        {n: len(v) for n, v in per_kernel.items()})
    fr, fk, fc = out["FETCH_SIZE"]
    wr, wk, _ = out["WRITE_SIZE"]
    total = 0.0
    print(f"calibration: copy of 256 MiB reads FETCH x {fr:.4f}, WRITE x {wr:.4f}")
    for n in sorted(fk):
        fb = fk[n] * fr * 1024
        wb = wk.get(n, 0.0) * wr * 1024
        total += fb + wb
        print(f"kernel: {n[:100]} | dispatches {fc[n]} | FETCH_SIZE {fk[n]:.0f} KiB | "
              f"WRITE_SIZE {wk.get(n, 0.0):.0f} KiB | HBM bytes {fb + wb:.0f}")
    print(f"hbm_bytes_per_launch: {total:.0f}")


def cpu_baseline(L):
    """The CPU oracle (fp64 numpy) on a bounded sample of the headline
    workload `L`: its first sequence (4096 tokens) as a one-sequence prefill,
    the whole layer, with BLAS threads set to every core of the affinity
    mask."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    cores = len(os.sched_getaffinity(0))
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    L = dict(L)
    T = L["cfg"]["T"]
    L["cfg"] = dict(L["cfg"], B=1)
    L["x"], L["psi"] = np.ascontiguousarray(L["x"][:T]), np.ascontiguousarray(L["psi"][:T])
    with threadpool_limits(limits=cores):
        t0 = time.perf_counter()
        oracle.layer_prefill(L)
        dt = time.perf_counter() - t0
    return {"value": round(T / dt, 2), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu_model": model,
            "sample": f"the first 4096-token sequence of the 1.3B-class prefill workload as a "
                      f"one-sequence layer (router, cache, attention, experts) through the "
                      f"fp64 oracle, {dt:.1f} s"}


if __name__ == "__main__":
    main()
