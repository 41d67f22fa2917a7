"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/triroute.h declares, and rejects bad arguments with
the documented status codes before launching anything."""
import ctypes as C
import os
import re

import pytest

import paper_2607_06601_amd as tr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    text = open(os.path.join(ROOT, "include", "triroute.h")).read()
    return sorted(set(re.findall(r"\b(triroute_[a-z_0-9]+)\s*\(", text)))


def cfg160(**over):
    c = tr.make_cfg(768, 12, 3, 64, 128, 8, 2, 2048, 64, "bf16")
    for k, v in over.items():
        setattr(c, k, v)
    return c


def test_library_exports_every_declared_symbol():
    lib = tr.lib()
    names = declared()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(tr.EXPORTS)


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 96, -2), ("kv_group", 48, -2), ("n_kv_heads", 5, -1), ("top_k", 10, -1),
    ("act", 7, -1), ("d_router", 64, -2), ("rms_eps", 0.0, -1), ("d_model", 100, -2),
    ("n_heads", 0, -1), ("d_psi", 6, -2), ("d_psi", 36, -2), ("attn_groups", 5, -1),
    ("attn_groups", -1, -1)])
def test_validate_rejects(field, value, code):
    assert tr.validate(cfg160(**{field: value})) == code
    assert tr.lib().triroute_last_error()


def test_validate_accepts_every_workload():
    import gen
    from paper_2607_06601_amd.device import cfg_from
    for name, shape in gen.CONFIGS.items():
        assert tr.validate(cfg_from(shape)) == 0, name
        for groups in (1, shape["Hkv"]):  # per-token and per-kv-group decisions
            assert tr.validate(cfg_from(dict(shape, attn_groups=groups))) == 0, (name, groups)


def test_workspace_and_cache_sizes():
    c = cfg160()
    # rotation table: (cos, sin) fp32 per token and pair (d_h / 2 = 32 pairs)
    assert tr.workspace_bytes(c, tr.OP_QKV, 8, 2048) == 8 * 2048 * 32 * 8
    # the per-row pool lengths before the append (rounded to 256 B)
    assert tr.workspace_bytes(c, tr.OP_KV_APPEND, 8, 2048) == 256
    lay = tr.workspace_bytes(c, tr.OP_LAYER_PREFILL, 8, 2048)
    assert lay > tr.workspace_bytes(c, tr.OP_MOE, 8, 2048)
    n = C.c_size_t()
    # 1.3B decode: dh 128, G 64: a 32-slot tile of one kv head holds 80/144/272/512 B per slot
    c5 = tr.make_cfg(2048, 16, 4, 128, 1024, 16, 2, 5632, 64, "bf16")
    assert tr.lib().triroute_kv_cache_bytes(C.byref(c5), 32, 32784, C.byref(n)) == 0
    tiles = (32784 + 31) // 32
    pools = 32 * 4 * tiles * 32 * (80 + 144 + 272 + 512)
    assert pools < n.value < pools + 32 * 16 * 32784 * 4 + (1 << 20)


def test_bad_calls_return_codes_without_launching():
    lib = tr.lib()
    c = cfg160()
    rw, cmp = tr.RouterW(), tr.Compaction()
    # NULL pointers
    r = lib.triroute_router(C.byref(c), 8, 2048, None, None, C.byref(rw), None, None, None,
                            None, None, C.byref(cmp), None, 0, None)
    assert r == tr.lib().triroute_validate(None) == -1
    # workspace too small (all pointers non-NULL but never dereferenced on the host)
    fake = 1 << 40
    rw = tr.RouterW(*([fake] * 12))
    cmp = tr.Compaction(*([fake] * 5))
    r = lib.triroute_router(C.byref(c), 8, 2048, fake, fake, C.byref(rw), fake, fake, fake,
                            fake, fake, C.byref(cmp), fake, 1024, None)
    assert r == -3 and b"workspace" in lib.triroute_last_error()
    # a tensor pointer off 16-byte alignment
    r = lib.triroute_router(C.byref(c), 8, 2048, fake + 8, fake, C.byref(rw), fake, fake, fake,
                            fake, fake, C.byref(cmp), fake, 1 << 40, None)
    assert r == -1 and b"aligned" in lib.triroute_last_error()
    dw = tr.DenseW(*([fake] * 5))
    r = lib.triroute_oproj(C.byref(c), 16, fake, fake + 2, C.byref(dw), fake, None)
    assert r == -1 and b"aligned" in lib.triroute_last_error()
    # B*T beyond the supported range
    n = C.c_size_t()
    assert lib.triroute_workspace_bytes(C.byref(c), 0, 1 << 13, 1 << 12, C.byref(n)) == -2
    # unknown op
    assert lib.triroute_workspace_bytes(C.byref(c), 42, 1, 1, C.byref(n)) == -1
    assert lib.triroute_status_string(-3) == b"workspace too small"


def test_relaxed_router_rejects_bad_parameters():
    """triroute_router_relaxed checks its relaxation parameters on the host
    (Sec. 3.4 temperatures, whitening statistics given together, the dual
    EMA momentum in [0, 1]) before anything is launched."""
    lib = tr.lib()
    c = cfg160()
    fake = 1 << 40
    rw = tr.RouterW(*([fake] * 12))
    cmp = tr.Compaction(*([fake] * 5))
    out = tr.RelaxOut(fake, fake, fake, fake, fake, None, None, None, None, None)

    def call(ws_bytes=1 << 40, **over):
        p = tr.RelaxParams(g_attn=fake, g_bits=fake, pos=fake, white_mu=fake, white_sd=fake,
                           white_eps=1e-5, tau_a=1.0, tau_b=1.0, zeta=0.5, alpha=0.01,
                           beta=0.001, gamma=0.1, dual=None, dual_lr=0.05, dual_ema=0.1)
        for k, v in over.items():
            setattr(p, k, v)
        return lib.triroute_router_relaxed(C.byref(c), 8, 2048, fake, fake, C.byref(rw),
                                           C.byref(p), fake, fake, fake, fake, fake,
                                           C.byref(cmp), C.byref(out), fake, ws_bytes, None)
    assert call(tau_a=0.0) == -1 and b"temperature" in lib.triroute_last_error()
    assert call(tau_b=float("inf")) == -1
    assert call(white_sd=None) == -1 and b"white_mu" in lib.triroute_last_error()
    assert call(g_bits=None) == -1
    assert call(dual_ema=1.5) == -1 and b"dual_ema" in lib.triroute_last_error()
    assert call(zeta=float("nan")) == -1
    assert call(ws_bytes=1024) == -3
    n = C.c_size_t()
    assert lib.triroute_workspace_bytes(C.byref(c), tr.OP_ROUTER_RELAXED, 8, 2048, C.byref(n)) == 0
    # beyond the router's scratch: the logits and h^ of every token
    assert n.value > tr.workspace_bytes(c, tr.OP_ROUTER, 8, 2048) + 8 * 2048 * (3 * 12 + 9 + 4 + 128) * 4


def test_relaxed_backward_rejects_bad_arguments():
    """triroute_router_relaxed_backward needs the forward's statistics and
    usage, the upstream gradients and a momentum in [0, 1]; checked on the
    host before any launch."""
    lib = tr.lib()
    c = cfg160()
    fake = 1 << 40
    rw = tr.RouterW(*([fake] * 12))
    p = tr.RelaxParams(pos=fake, tau_a=1.0, tau_b=1.0, zeta=0.5, alpha=0.01, beta=0.001,
                       gamma=0.1)
    go = tr.RelaxGradOut(*([fake] * 14), None)

    def call(fwd_usage=fake, g_gate=fake, rho_m=0.1, ws_bytes=1 << 40, dx=fake):
        fwd = tr.RelaxOut(y_attn=fake, y_bits=fake, stats=fake, usage_exp=fwd_usage)
        gin = tr.RelaxGradIn(g_attn=fake, g_bits=fake, g_gate=g_gate, rho_m=rho_m)
        go.dx = dx
        return lib.triroute_router_relaxed_backward(C.byref(c), 8, 2048, fake, fake, C.byref(rw),
                                                    C.byref(p), C.byref(fwd), fake, fake,
                                                    C.byref(gin), C.byref(go), fake, ws_bytes, None)
    assert call(fwd_usage=None) == -1 and b"usage_exp" in lib.triroute_last_error()
    assert call(g_gate=None) == -1 and b"upstream" in lib.triroute_last_error()
    assert call(rho_m=2.0) == -1 and b"rho_m" in lib.triroute_last_error()
    assert call(dx=fake + 4) == -1 and b"aligned" in lib.triroute_last_error()
    assert call(ws_bytes=1024) == -3
    assert tr.workspace_bytes(c, tr.OP_ROUTER_RELAXED_BACKWARD, 8, 2048) > \
        tr.workspace_bytes(c, tr.OP_ROUTER_RELAXED, 8, 2048)


def test_paged_cache_sizes_and_rejections():
    """A paged cache sized for the pages the workload's widths need is far
    smaller than one that reserves the capacity in every width pool; bad
    page arguments are refused on the host."""
    lib = tr.lib()
    c = tr.make_cfg(2048, 16, 4, 128, 1024, 16, 2, 5632, 64, "bf16")
    n = C.c_size_t()
    pages = (C.c_int32 * 4)(740, 215, 4, 110)  # 32 sequences of 32768 slots at 70/20/0/10 %
    assert lib.triroute_kv_paged_cache_bytes(C.byref(c), 32, 32784, 32, pages, C.byref(n)) == 0
    paged = n.value
    assert lib.triroute_kv_cache_bytes(C.byref(c), 32, 32784, C.byref(n)) == 0
    assert paged < n.value / 6
    bad = (C.c_int32 * 4)(1, -1, 1, 1)
    assert lib.triroute_kv_paged_cache_bytes(C.byref(c), 32, 32784, 32, bad, C.byref(n)) == -1
    assert lib.triroute_kv_paged_cache_bytes(C.byref(c), 32, 32784, 0, pages, C.byref(n)) == -1
    assert lib.triroute_kv_paged_cache_bytes(C.byref(c), 32, 32784, 32, None, C.byref(n)) == -1
    desc = tr.KVCacheDesc()
    desc.base = 1 << 40
    out = (C.c_int32 * 4)()
    assert lib.triroute_kv_free_pages(C.byref(desc), out, None) == -1  # not paged
    assert b"not paged" in lib.triroute_last_error()
