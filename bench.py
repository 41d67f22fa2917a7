"""Benchmark of the TriRoute routed-layer forward on one MI355X.

A step is one full routed-layer prefill (router, compaction, QKV + RoPE,
KV quantize/append, attention, O-proj, second norm, expert grouped GEMM,
combine) of the 160M-class workload: batch 8 x 2048 tokens, d 768, 12 x 64
heads (3 kv heads), window 128, 8 SwiGLU experts (d_ff 2048) + null, top-2,
KV group 64, bf16, seeded synthetic inputs and random-init weights.  Inputs
are resident in HBM before timing; every step writes a fresh cache; the
L2 / Infinity Cache is flushed before each timed step by reading a 1 GiB
buffer (a read, so that no dirty lines are left whose write-back would land
in the timed region).

Also reported: the MoE sublayer's achieved bf16 MFMA rate (roofline), the
410M-class decode step (64 sequences x 8192 context) and its decode
attention's achieved HBM bandwidth, and the CPU oracle timed on a bounded
sample on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2516.6  # MI355X dense bf16 MFMA, TFLOP/s (256 CU x 2.4 GHz x 4096)

PREFILL = "160m_bf16_prefill"
DECODE = "410m_bf16_decode"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-decode", action="store_true")
    p.add_argument("--no-wide", action="store_true",
                   help="leave out the 1.3B-class prefill and long-context decode legs")
    p.add_argument("--only", choices=("prefill", "decode", "moe", "prefill_1p3b", "decode_1p3b"),
                   default=None,
                   help="profile one workload alone (prints its section only); 'moe' times "
                        "the MoE sublayer and then runs a 256 MiB copy for counter calibration")
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


def events(torch):
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the routed layer is "
              "measured on a single MI355X in this build", file=sys.stderr)
        sys.exit(2)
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc)
        return
    import numpy as np
    import torch

    import gen
    import paper_2607_06601_amd as tr
    from paper_2607_06601_amd.device import DeviceLayer, to_dev

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    tr.lib()
    dev = "cuda"
    stream = torch.cuda.current_stream()
    flush = CacheFlush(torch, dev)
    if args.only == "decode":
        res = bench_decode(args, torch, np, gen, tr, DeviceLayer, to_dev, flush, DECODE)
        copy_calibration(torch)
        print(json.dumps({"decode": res}), flush=True)
        return
    if args.only in ("prefill_1p3b", "decode_1p3b"):
        res = run_wide(args, torch, np, gen, tr, DeviceLayer, to_dev, flush, args.only)
        print(json.dumps({args.only: res}), flush=True)
        return

    res = bench_prefill(args, torch, np, gen, tr, DeviceLayer, flush, PREFILL, 1)
    if args.only == "moe":
        copy_calibration(torch)
        print(json.dumps({"moe": res["roofline"]}), flush=True)
        return
    B, T, ms, step_ms, wall = (res[x] for x in ("B", "T", "ms", "step_ms", "wall"))
    N = B * T
    roofline = res["roofline"]

    out = {
        "metric": "routed-layer tokens/s (prefill, decode); decode-attn HBM GB/s; MoE MFMA util",
        "value": round(N / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded generator, random-init weights)",
        "config": {"workload": "160M-class TriRoute layer prefill: batch 8 x seq 2048, d 768, "
                               "12x64 heads (3 kv), window 128, 8 SwiGLU experts d_ff 2048 + "
                               "null, top-2, KV group 64, bf16",
                   "global_batch": B, "seq_len": T, "parallelism": "single GPU"},
        "roofline": roofline,
        "timing": {"per_step_ms_min": round(min(step_ms), 4),
                   "per_step_ms_max": round(max(step_ms), 4),
                   "wall_s_timed_loop": round(wall, 3), "cache_flush_per_step": "1 GiB read"},
    }

    # ------------------------------------------------------------- decode
    if not args.no_decode and args.only is None:
        out["decode"] = bench_decode(args, torch, np, gen, tr, DeviceLayer, to_dev, flush, DECODE)

    # ---------------------------------- the 1.3B-class workloads (context)
    if not args.no_wide and args.only is None:
        for leg in ("prefill_1p3b", "decode_1p3b"):
            out[leg] = run_wide(args, torch, np, gen, tr, DeviceLayer, to_dev, flush, leg)

    # --------------------------------------------------------- CPU oracle
    if not args.no_cpu_baseline and args.only is None:
        out["cpu_baseline"] = cpu_baseline(np)
    print(json.dumps(out), flush=True)


def describe(cfg):
    """The workload's sizes in words."""
    if cfg["kind"] == "prefill":
        head = f"layer prefill: batch {cfg['B']} x seq {cfg['T']}"
    else:
        head = (f"decode step: {cfg['B']} sequences x 1 new token, context {cfg['ctx']} (bits "
                + "/".join(f"{round(100 * f)}" for f in cfg["ctx_bits"]) + " % for 2/4/8/16)")
    ex = "skewed" if cfg["experts"] == "skewed" else "uniform"
    return (f"{head}, d {cfg['d']}, {cfg['H']}x{cfg['dh']} heads ({cfg['Hkv']} kv), window "
            f"{cfg['w']}, {cfg['E']} SwiGLU experts d_ff {cfg['d_ff']} + null, top-{cfg['k']} "
            f"({ex} routing), KV group {cfg['G']}, {cfg['act']}")


def run_wide(args, torch, np, gen, tr, DeviceLayer, to_dev, flush, leg):
    """The 1.3B-class prefill (step + MoE sublayer) or long-context decode
    (step + decode attention), with at most 10 timed steps."""
    import copy
    a = copy.copy(args)
    a.steps, a.warmup = min(args.steps, 10), min(args.warmup, 3)
    if leg == "prefill_1p3b":
        name = "1p3b_bf16_prefill"
        r = bench_prefill(a, torch, np, gen, tr, DeviceLayer, flush, name, None)
        N = r["B"] * r["T"]
        return {"workload": "1.3B-class " + describe(gen.CONFIGS[name]),
                "tokens_per_s": round(N / (r["ms"] * 1e-3), 1), "ms_per_step": round(r["ms"], 4),
                "steps": a.steps, "moe": r["roofline"]}
    return bench_decode(a, torch, np, gen, tr, DeviceLayer, to_dev, flush, "1p3b_bf16_decode")


def bench_prefill(args, torch, np, gen, tr, DeviceLayer, flush, name, seed):
    """Timed triroute_layer_prefill steps of one prefill workload, then its
    MoE sublayer alone on the same routed inputs."""
    L = gen.make_layer(name, seed)
    cfg = L["cfg"]
    B, T, d, k = (cfg[x] for x in ("B", "T", "d", "k"))
    N = B * T
    D = DeviceLayer(L)
    del L
    c = D.cfg
    dev = "cuda"
    stream = torch.cuda.current_stream()
    ws = tr.workspace(c, tr.OP_LAYER_PREFILL, B, T)
    xo = torch.empty(N, d, dtype=D.act, device=dev)
    caches = [tr.KVCache(c, B, T) for _ in range(args.steps)]
    warm = tr.KVCache(c, B, T)
    eidx_t = torch.empty(N, k, dtype=torch.int32, device=dev)
    egate_t = torch.empty(N, k, dtype=torch.float32, device=dev)
    xt_t = torch.empty(N, d, dtype=D.act, device=dev)
    taps = tr.Taps(eidx=eidx_t.data_ptr(), egate=egate_t.data_ptr(), xt=xt_t.data_ptr())
    for _ in range(args.warmup):
        for s in range(B):
            warm.reset_seq(s)
        tr.layer_prefill(c, B, T, D.x, D.psi, D.rw, D.dw, D.mw, warm, xo, ws, taps=taps)
    torch.cuda.synchronize()
    times = []
    t_wall0 = time.perf_counter()
    for i in range(args.steps):
        flush()
        e0, e1 = events(torch)
        e0.record(stream)
        tr.layer_prefill(c, B, T, D.x, D.psi, D.rw, D.dw, D.mw, caches[i], xo, ws, taps=taps)
        e1.record(stream)
        times.append((e0, e1))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall0
    step_ms = [a.elapsed_time(b) for a, b in times]
    for cc in caches:
        assert cc.status() == 0
    del caches, warm
    roofline = bench_moe(args, torch, np, tr, D, c, B, T, flush, eidx_t, egate_t, xt_t, xo,
                         name)
    return {"B": B, "T": T, "ms": float(np.mean(step_ms)), "step_ms": step_ms, "wall": wall,
            "roofline": roofline}


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


def bench_moe(args, torch, np, tr, D, c, B, T, flush, eidx_t, egate_t, xt_t, xo, name):
    """The MoE sublayer (triroute_moe: rmsnorm2, grouped GEMM gate/up + SwiGLU,
    grouped GEMM down, combine) alone on the routed inputs of the last prefill
    step: achieved bf16 MFMA rate of the expert FLOPs."""
    dev = "cuda"
    stream = torch.cuda.current_stream()
    d, dff = c.d_model, c.d_ff
    N = B * T
    eidx_h = eidx_t.cpu().numpy()
    n_real = int((eidx_h != 0).sum())
    moe_flops = 6.0 * d * dff * n_real
    cmp = tr.CompactionBuffers(c, B, T)
    rw_ws = tr.workspace(c, tr.OP_ROUTER, B, T)
    n1 = torch.empty(N, d, dtype=D.act, device=dev)
    mode = torch.empty(N, c.n_heads, dtype=torch.uint8, device=dev)
    bit = torch.empty(N, dtype=torch.uint8, device=dev)
    tr.router(c, B, T, D.x, D.psi, D.rw, n1, mode, bit, eidx_t, egate_t, cmp.struct, rw_ws)
    moe_ws = tr.workspace(c, tr.OP_MOE, N, 1)
    for _ in range(3):
        tr.moe(c, N, xt_t, D.dw, D.mw, eidx_t, egate_t, cmp.struct, xo, moe_ws)
    moe_ms = []
    for i in range(args.steps):
        flush()
        e0, e1 = events(torch)
        e0.record(stream)
        tr.moe(c, N, xt_t, D.dw, D.mw, eidx_t, egate_t, cmp.struct, xo, moe_ws)
        e1.record(stream)
        moe_ms.append((e0, e1))
    torch.cuda.synchronize()
    moe_avg = float(np.mean([a.elapsed_time(b) for a, b in moe_ms]))
    moe_tflops = moe_flops / (moe_avg * 1e-3) / 1e12
    return {"kernel": "triroute_moe (rmsnorm2, grouped GEMM gate/up + SwiGLU, grouped GEMM "
                      "down, combine)",
            "bound": "mfma", "achieved": round(moe_tflops, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(moe_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": (stored_traffic("moe_160m_prefill_traffic.txt", MOE_SOURCES)
                        if name == PREFILL else None),
            "algorithmic": f"6*d*d_ff FLOP x {n_real} real assignments = "
                           f"{moe_flops / 1e9:.1f} GFLOP per launch",
            "avg_ms": round(moe_avg, 4)}


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


def decode_attn_bytes(cfg, mode, bits_per_seq):
    """Algorithmic bytes the routed decode attention must read: per (sequence,
    kv head), the union of the key ranges its query heads need (full -> all
    P+1 keys, local -> last w, skip -> none) x packed K+V bytes incl. fp16
    scale/zero."""
    import numpy as np
    H, Hkv, dh, G, w = cfg["H"], cfg["Hkv"], cfg["dh"], cfg["G"], cfg["w"]
    grp = H // Hkv
    per_tok = np.array([2 * dh * b / 8 + (2 * (dh // G) * 4 if b < 16 else 0)
                        for b in (2, 4, 8, 16)])
    total = 0.0
    for s, bits in enumerate(bits_per_seq):
        P1 = len(bits)
        full_b = per_tok[bits].sum()
        loc_b = per_tok[bits[max(0, P1 - w):]].sum()
        for g in range(Hkv):
            m = mode[s, g * grp:(g + 1) * grp].max()
            total += full_b if m == 2 else loc_b if m == 1 else 0.0
    return total


def bench_decode(args, torch, np, gen, tr, DeviceLayer, to_dev, flush, name):
    L = gen.make_layer(name)
    cfg = L["cfg"]
    B, ctx, d, H, k = cfg["B"], cfg["ctx"], cfg["d"], cfg["H"], cfg["k"]
    D = DeviceLayer(L)
    c = D.cfg
    dev = "cuda"
    stream = torch.cuda.current_stream()
    cap = ctx + args.warmup + args.steps + 1
    cache = tr.KVCache(c, B, cap)
    ws_app = tr.workspace(c, tr.OP_KV_APPEND, 1, ctx)
    bits_all = []
    for s in range(B):
        kk, vv = gen.context_kv(cfg, s)
        bits = gen.context_bits(cfg, s)
        bits_all.append(bits)
        tr.kv_append(c, cache, 1, ctx, to_dev(kk.reshape(ctx, -1), D.act),
                     to_dev(vv.reshape(ctx, -1), D.act), to_dev(bits, torch.uint8), ws_app,
                     seq_ids=torch.tensor([s], dtype=torch.int32, device=dev))
    torch.cuda.synchronize()
    ws = tr.workspace(c, tr.OP_LAYER_DECODE, B, 1)
    xo = torch.empty(B, d, dtype=D.act, device=dev)
    mode_t = torch.empty(B, H, dtype=torch.uint8, device=dev)
    bit_t = torch.empty(B, dtype=torch.uint8, device=dev)
    q_t = torch.empty(B, H * cfg["dh"], dtype=D.act, device=dev)
    taps = tr.Taps(mode=mode_t.data_ptr(), bit=bit_t.data_ptr(), q=q_t.data_ptr())
    for _ in range(args.warmup):
        tr.layer_decode(c, B, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo, ws, taps=taps)
    times = []
    for i in range(args.steps):
        flush()
        e0, e1 = events(torch)
        e0.record(stream)
        tr.layer_decode(c, B, D.x, D.psi, D.rw, D.dw, D.mw, cache, xo, ws, taps=taps)
        e1.record(stream)
        times.append((e0, e1))
    torch.cuda.synchronize()
    assert cache.status() == 0
    step_ms = float(np.mean([a.elapsed_time(b) for a, b in times]))
    # decode attention alone over the cache as it now stands
    mode = mode_t.cpu().numpy()
    seq_len = cache.seq_len().cpu().numpy()
    # bit widths of every cached token, in position order, per sequence
    extra = bit_t.cpu().numpy()
    bits_now = [np.concatenate([bits_all[s], np.full(seq_len[s] - ctx, extra[s], np.uint8)])
                for s in range(B)]
    nbytes = decode_attn_bytes(cfg, mode, bits_now)
    o = torch.empty(B, H * cfg["dh"], dtype=D.act, device=dev)
    aws = tr.workspace(c, tr.OP_ATTN_DECODE, B, 1)
    for _ in range(3):
        tr.attn_decode(c, B, q_t, cache, mode_t, o, aws)
    at = []
    for i in range(args.steps):
        flush()
        e0, e1 = events(torch)
        e0.record(stream)
        tr.attn_decode(c, B, q_t, cache, mode_t, o, aws)
        e1.record(stream)
        at.append((e0, e1))
    torch.cuda.synchronize()
    attn_ms = float(np.mean([a.elapsed_time(b) for a, b in at]))
    gbs = nbytes / (attn_ms * 1e-3) / 1e9
    cls = "410M" if name == DECODE else "1.3B"
    return {"workload": f"{cls}-class " + describe(cfg),
            "tokens_per_s": round(B / (step_ms * 1e-3), 1), "ms_per_step": round(step_ms, 4),
            "attn": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "algorithmic_bytes": int(nbytes), "avg_ms": round(attn_ms, 4),
                     "traffic": (stored_traffic("attn_decode_410m_traffic.txt",
                                                 DECODE_ATTN_SOURCES) if name == DECODE else None)}}


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


def cpu_baseline(np):
    """The CPU oracle (fp64 numpy) on the whole prefill workload (8 x 2048
    tokens), on the host cores."""
    import gen
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    L = gen.make_layer(PREFILL, 1)
    N = L["cfg"]["B"] * L["cfg"]["T"]
    t0 = time.perf_counter()
    oracle.layer_prefill(L)
    dt = time.perf_counter() - t0
    return {"value": round(N / dt, 2), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"the whole prefill workload (8 x 2048 tokens) through the fp64 oracle, "
                      f"{dt:.1f} s"}


if __name__ == "__main__":
    main()
