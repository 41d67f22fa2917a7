"""Python binding of libtriroute: the TriRoute routed-layer forward on MI355X.

Argument marshalling only.  Every stage runs in the HIP kernels of
``libtriroute.so`` (built from ``csrc/`` for gfx950); PyTorch supplies device
memory (``tensor.data_ptr()``) and the current HIP stream.  There is no CPU
path: importing succeeds without the library, but every call raises if it is
missing.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtriroute.so")

F32, BF16 = 0, 1
SKIP, LOCAL, FULL = 0, 1, 2
OP_ROUTER, OP_QKV, OP_KV_APPEND, OP_ATTN_PREFILL, OP_ATTN_DECODE, OP_MOE, \
    OP_LAYER_PREFILL, OP_LAYER_DECODE, OP_STACK_DECODE, OP_ROUTER_RELAXED, \
    OP_ROUTER_RELAXED_BACKWARD = range(11)
# fp64 fields of RelaxOut.stats (axes in the order attention, experts, bits)
RS_LBAL, RS_LZ, RS_LENT, RS_ENTROPY, RS_CBAR, RS_COST, RS_DENSE, RS_REG = 0, 3, 6, 9, 12, 14, 16, 18
RS_F_ATTN, RS_P_ATTN, RS_F_BITS, RS_P_BITS, RELAX_NSTAT = 19, 22, 25, 29, 33
CACHE_OVERFLOW, CACHE_BAD_SEQ = 1, 2

STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported", -3: "workspace too small",
          -4: "cache capacity exceeded", -5: "HIP runtime error"}


class TrirouteError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)} ({status}): {msg}")
        self.status = status


# ------------------------------------------------------------------ structs
class Cfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "d_model", "n_heads", "n_kv_heads", "head_dim", "window", "n_experts", "top_k",
        "d_ff", "kv_group", "d_psi", "d_router", "act")] + [
        ("rms_eps", C.c_float), ("rope_theta", C.c_float), ("attn_groups", C.c_int32)]


class RouterW(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in
                ("g1", "W1", "b1", "W2", "b2", "gr", "Wa", "ca", "We", "ce", "Wb", "cb")]


class DenseW(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("Wq", "Wk", "Wv", "Wo", "g2")]


class MoeW(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("Wgate", "Wup", "Wdown")]


class LayerW(C.Structure):
    _fields_ = [("router", RouterW), ("dense", DenseW), ("moe", MoeW)]


class Compaction(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in
                ("attn_cnt", "attn_idx", "exp_cnt", "exp_off", "exp_rows")]


class KVCacheDesc(C.Structure):
    _fields_ = [("base", C.c_void_p), ("n_seq", C.c_int32), ("capacity", C.c_int32),
                ("tile_slots", C.c_int32), ("n_tiles", C.c_int32),
                ("off_status", C.c_int64), ("off_seq_len", C.c_int64),
                ("off_pool_len", C.c_int64), ("off_pos", C.c_int64),
                ("off_pool", C.c_int64 * 4), ("tile_bytes", C.c_int64 * 4),
                ("total_bytes", C.c_int64), ("page_tiles", C.c_int32), ("max_pages", C.c_int32),
                ("n_pages", C.c_int32 * 4), ("off_alloc", C.c_int64),
                ("off_page_table", C.c_int64), ("off_free_top", C.c_int64),
                ("off_free_list", C.c_int64 * 4), ("off_pos_pool", C.c_int64 * 4)]


class Taps(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in
                ("n1", "mode", "bit", "eidx", "egate", "q", "k", "v", "o", "xt")]


class RelaxParams(C.Structure):
    _fields_ = [("g_attn", C.c_void_p), ("g_bits", C.c_void_p), ("pos", C.c_void_p),
                ("white_mu", C.c_void_p), ("white_sd", C.c_void_p), ("white_eps", C.c_float),
                ("tau_a", C.c_float), ("tau_b", C.c_float), ("zeta", C.c_float),
                ("alpha", C.c_float), ("beta", C.c_float), ("gamma", C.c_float),
                ("c_target", C.c_float * 2), ("dual", C.c_void_p), ("dual_lr", C.c_float),
                ("dual_ema", C.c_float)]


class RelaxOut(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in
                ("y_attn", "y_bits", "c_flops", "c_mem", "stats", "p_exp", "usage_exp",
                 "h_mean", "h_var", "z")]


class RelaxGradIn(C.Structure):
    _fields_ = [("g_attn", C.c_void_p), ("g_bits", C.c_void_p), ("g_gate", C.c_void_p),
                ("lambda_", C.c_void_p), ("rho", C.c_void_p), ("rho_m", C.c_float)]


class RelaxGradOut(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in
                ("dW1", "db1", "dW2", "db2", "dgr", "dWa", "dca", "dWe", "dce", "dWb", "dcb",
                 "dg1", "dx", "dpsi", "lm_norm")]


EXPORTS = [
    "triroute_validate", "triroute_status_string", "triroute_last_error",
    "triroute_workspace_bytes", "triroute_kv_cache_bytes", "triroute_kv_cache_init",
    "triroute_kv_reset_seq", "triroute_kv_status", "triroute_kv_seq_len_ptr",
    "triroute_kv_append", "triroute_kv_export", "triroute_router", "triroute_qkv",
    "triroute_attn_prefill", "triroute_attn_decode", "triroute_oproj", "triroute_moe",
    "triroute_layer_prefill", "triroute_layer_decode", "triroute_layer_decode_noalloc",
    "triroute_stack_decode", "triroute_router_relaxed", "triroute_router_relaxed_backward",
    "triroute_kv_paged_cache_bytes", "triroute_kv_paged_cache_init", "triroute_kv_free_pages",
]

_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_06601_amd._build`")
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        i32, sz = C.c_int, C.c_size_t
        sig = {
            "triroute_validate": [P],
            "triroute_workspace_bytes": [P, i32, i32, i32, C.POINTER(sz)],
            "triroute_kv_cache_bytes": [P, i32, i32, C.POINTER(sz)],
            "triroute_kv_cache_init": [P, P, P, sz, i32, i32, P],
            "triroute_kv_paged_cache_bytes": [P, i32, i32, i32, P, C.POINTER(sz)],
            "triroute_kv_paged_cache_init": [P, P, P, sz, i32, i32, i32, P, P],
            "triroute_kv_free_pages": [P, P, P],
            "triroute_kv_reset_seq": [P, P, i32, P],
            "triroute_kv_status": [P, C.POINTER(C.c_int32), P],
            "triroute_kv_seq_len_ptr": [P],
            "triroute_kv_append": [P, P, i32, i32, P, P, P, P, P, sz, P],
            "triroute_kv_export": [P, P, i32, i32, i32, i32, P, P, P, P, P, P],
            "triroute_router": [P, i32, i32, P, P, P, P, P, P, P, P, P, P, sz, P],
            "triroute_qkv": [P, i32, i32, P, P, P, P, P, P, P, sz, P],
            "triroute_attn_prefill": [P, i32, i32, P, P, P, P, P, P, P, sz, P],
            "triroute_attn_decode": [P, i32, P, P, P, P, P, P, sz, P],
            "triroute_oproj": [P, i32, P, P, P, P, P],
            "triroute_moe": [P, i32, P, P, P, P, P, P, P, P, sz, P],
            "triroute_layer_prefill": [P, i32, i32, P, P, P, P, P, P, P, P, P, P, sz, P],
            "triroute_layer_decode": [P, i32, P, P, P, P, P, P, P, P, P, P, sz, P],
            "triroute_layer_decode_noalloc": [P, i32, P, P, P, P, P, P, P, P, P, P],
            "triroute_stack_decode": [P, i32, i32, P, P, P, P, P, P, P, sz, P],
            "triroute_router_relaxed": [P, i32, i32, P, P, P, P, P, P, P, P, P, P, P, P, sz, P],
            "triroute_router_relaxed_backward": [P, i32, i32, P, P, P, P, P, P, P, P, P, P, sz, P],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = C.c_int
        L.triroute_kv_seq_len_ptr.restype = C.c_void_p
        L.triroute_status_string.restype = C.c_char_p
        L.triroute_status_string.argtypes = [C.c_int]
        L.triroute_last_error.restype = C.c_char_p
        L.triroute_last_error.argtypes = []
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise TrirouteError(status, lib().triroute_last_error().decode())


def _p(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def act_dtype(cfg: Cfg):
    return torch.bfloat16 if cfg.act == BF16 else torch.float32


def make_cfg(d_model, n_heads, n_kv_heads, head_dim, window, n_experts, top_k, d_ff,
             kv_group, act, d_psi=8, d_router=128, rms_eps=1e-6, rope_theta=1e4,
             attn_groups=0) -> Cfg:
    return Cfg(d_model, n_heads, n_kv_heads, head_dim, window, n_experts, top_k, d_ff,
               kv_group, d_psi, d_router, BF16 if act in ("bf16", BF16) else F32,
               rms_eps, rope_theta, attn_groups)


def validate(cfg: Cfg) -> int:
    return lib().triroute_validate(C.byref(cfg))


def workspace_bytes(cfg: Cfg, op: int, B: int, T: int) -> int:
    n = C.c_size_t()
    _check(lib().triroute_workspace_bytes(C.byref(cfg), op, B, T, C.byref(n)))
    return n.value


def workspace(cfg: Cfg, op: int, B: int, T: int, device="cuda"):
    n = workspace_bytes(cfg, op, B, T)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


# ------------------------------------------------------------------ cache
class KVCache:
    """A device allocation laid out by triroute_kv_cache_init, or, with
    ``pages=(page_tiles, [n_pages per width])``, by triroute_kv_paged_cache_init."""

    def __init__(self, cfg: Cfg, n_seq: int, capacity: int, device="cuda", stream=None,
                 pages=None):
        n = C.c_size_t()
        self.cfg = cfg
        self.desc = KVCacheDesc()
        if pages is None:
            _check(lib().triroute_kv_cache_bytes(C.byref(cfg), n_seq, capacity, C.byref(n)))
        else:
            pt, npg = pages
            self._np = (C.c_int32 * 4)(*npg)
            _check(lib().triroute_kv_paged_cache_bytes(C.byref(cfg), n_seq, capacity, pt, self._np,
                                                       C.byref(n)))
        self.nbytes = n.value
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        if pages is None:
            _check(lib().triroute_kv_cache_init(C.byref(cfg), C.byref(self.desc),
                                                self.buf.data_ptr(), self.nbytes, n_seq,
                                                capacity, _stream(stream)))
        else:
            _check(lib().triroute_kv_paged_cache_init(C.byref(cfg), C.byref(self.desc),
                                                      self.buf.data_ptr(), self.nbytes, n_seq,
                                                      capacity, pt, self._np, _stream(stream)))

    def free_pages(self, stream=None):
        out = (C.c_int32 * 4)()
        _check(lib().triroute_kv_free_pages(self.ref, out, _stream(stream)))
        return list(out)

    @property
    def ref(self):
        return C.byref(self.desc)

    def seq_len_ptr(self) -> int:
        return lib().triroute_kv_seq_len_ptr(self.ref)

    def _meta(self, off, count):
        return self.buf[off:off + 4 * count].view(torch.int32)

    def seq_len(self):
        return self._meta(self.desc.off_seq_len, self.desc.n_seq)

    def pool_len(self):
        return self._meta(self.desc.off_pool_len, 4 * self.desc.n_seq).view(-1, 4)

    def status(self, stream=None) -> int:
        s = C.c_int32()
        _check(lib().triroute_kv_status(self.ref, C.byref(s), _stream(stream)))
        return s.value

    def reset_seq(self, seq: int, stream=None):
        _check(lib().triroute_kv_reset_seq(C.byref(self.cfg), self.ref, seq, _stream(stream)))


# ------------------------------------------------------------ per-stage calls
def kv_append(cfg, cache: KVCache, B, T, k, v, bit, ws, seq_ids=None, stream=None):
    _check(lib().triroute_kv_append(C.byref(cfg), cache.ref, B, T, _p(seq_ids), _p(k), _p(v),
                                    _p(bit), _p(ws), ws.numel() if ws is not None else 0,
                                    _stream(stream)))


def kv_export(cfg, cache: KVCache, seq, bi, slot0, count, k_out, v_out, k_sz=None, v_sz=None,
              pos_out=None, stream=None):
    _check(lib().triroute_kv_export(C.byref(cfg), cache.ref, seq, bi, slot0, count, _p(k_out),
                                    _p(v_out), _p(k_sz), _p(v_sz), _p(pos_out),
                                    _stream(stream)))


def router(cfg, B, T, x, psi, rw: RouterW, n1, mode, bit, eidx, egate, cmp: Compaction, ws,
           stream=None):
    _check(lib().triroute_router(C.byref(cfg), B, T, _p(x), _p(psi), C.byref(rw), _p(n1),
                                 _p(mode), _p(bit), _p(eidx), _p(egate), C.byref(cmp), _p(ws),
                                 ws.numel(), _stream(stream)))


def router_relaxed(cfg, B, T, x, psi, rw: RouterW, params: RelaxParams, n1, mode, bit, eidx,
                   egate, cmp: Compaction, out: RelaxOut, ws, stream=None):
    """Training-time relaxed controller forward (triroute_router_relaxed)."""
    _check(lib().triroute_router_relaxed(C.byref(cfg), B, T, _p(x), _p(psi), C.byref(rw),
                                         C.byref(params), _p(n1), _p(mode), _p(bit), _p(eidx),
                                         _p(egate), C.byref(cmp), C.byref(out), _p(ws),
                                         ws.numel(), _stream(stream)))


def router_relaxed_backward(cfg, B, T, x, psi, rw: RouterW, params: RelaxParams,
                            fwd: RelaxOut, eidx, egate, gin: RelaxGradIn, gout: RelaxGradOut, ws,
                            stream=None):
    """Backward pass of the relaxed controller (triroute_router_relaxed_backward)."""
    _check(lib().triroute_router_relaxed_backward(
        C.byref(cfg), B, T, _p(x), _p(psi), C.byref(rw), C.byref(params), C.byref(fwd), _p(eidx),
        _p(egate), C.byref(gin), C.byref(gout), _p(ws), ws.numel(), _stream(stream)))


def qkv(cfg, B, T, n1, dw: DenseW, q, k, v, ws, pos0=None, stream=None):
    _check(lib().triroute_qkv(C.byref(cfg), B, T, _p(n1), C.byref(dw), _p(pos0), _p(q), _p(k),
                              _p(v), _p(ws), ws.numel(), _stream(stream)))


def attn_prefill(cfg, B, T, q, cache: KVCache, mode, cmp: Compaction, o, ws=None,
                 seq_ids=None, stream=None):
    _check(lib().triroute_attn_prefill(C.byref(cfg), B, T, _p(seq_ids), _p(q), cache.ref,
                                       _p(mode), C.byref(cmp), _p(o), _p(ws),
                                       ws.numel() if ws is not None else 0, _stream(stream)))


def attn_decode(cfg, B, q, cache: KVCache, mode, o, ws=None, seq_ids=None, stream=None):
    _check(lib().triroute_attn_decode(C.byref(cfg), B, _p(seq_ids), _p(q), cache.ref, _p(mode),
                                      _p(o), _p(ws), ws.numel() if ws is not None else 0,
                                      _stream(stream)))


def oproj(cfg, n_tok, x, o, dw: DenseW, xt, stream=None):
    _check(lib().triroute_oproj(C.byref(cfg), n_tok, _p(x), _p(o), C.byref(dw), _p(xt),
                                _stream(stream)))


def moe(cfg, n_tok, xt, dw: DenseW, mw: MoeW, eidx, egate, cmp: Compaction, x_out, ws,
        stream=None):
    _check(lib().triroute_moe(C.byref(cfg), n_tok, _p(xt), C.byref(dw), C.byref(mw), _p(eidx),
                              _p(egate), C.byref(cmp), _p(x_out), _p(ws), ws.numel(),
                              _stream(stream)))


def layer_prefill(cfg, B, T, x, psi, rw, dw, mw, cache: KVCache, x_out, ws, taps=None,
                  seq_ids=None, stream=None):
    _check(lib().triroute_layer_prefill(
        C.byref(cfg), B, T, _p(seq_ids), _p(x), _p(psi), C.byref(rw), C.byref(dw), C.byref(mw),
        cache.ref, _p(x_out), C.byref(taps) if taps is not None else None, _p(ws), ws.numel(),
        _stream(stream)))


def layer_decode(cfg, B, x, psi, rw, dw, mw, cache: KVCache, x_out, ws, taps=None,
                 seq_ids=None, stream=None):
    _check(lib().triroute_layer_decode(
        C.byref(cfg), B, _p(seq_ids), _p(x), _p(psi), C.byref(rw), C.byref(dw), C.byref(mw),
        cache.ref, _p(x_out), C.byref(taps) if taps is not None else None, _p(ws), ws.numel(),
        _stream(stream)))


def layer_decode_noalloc(cfg, B, x, psi, rw, dw, mw, cache: KVCache, x_out, taps=None,
                         seq_ids=None, stream=None):
    """triroute_layer_decode with the library's static scratch (no workspace)."""
    _check(lib().triroute_layer_decode_noalloc(
        C.byref(cfg), B, _p(seq_ids), _p(x), _p(psi), C.byref(rw), C.byref(dw), C.byref(mw),
        cache.ref, _p(x_out), C.byref(taps) if taps is not None else None, _stream(stream)))


def stack_decode(cfg, B, x, psi, layers, caches, x_out, ws, seq_ids=None, stream=None):
    """One decode step through len(layers) routed layers; ``layers`` is a list
    of (RouterW, DenseW, MoeW), ``caches`` one KVCache per layer."""
    n = len(layers)
    lw = (LayerW * n)(*[LayerW(r, d, m) for r, d, m in layers])
    cs = (type(caches[0].desc) * n)(*[c.desc for c in caches])
    _check(lib().triroute_stack_decode(
        C.byref(cfg), n, B, _p(seq_ids), _p(x), _p(psi), lw, cs, _p(x_out), _p(ws), ws.numel(),
        _stream(stream)))


# ------------------------------------------------------ device-side buffers
class CompactionBuffers:
    """Device arrays of one compaction (owned by torch)."""

    def __init__(self, cfg: Cfg, B: int, T: int, device="cuda"):
        H, E, k = cfg.n_heads, cfg.n_experts, cfg.top_k
        i32 = dict(dtype=torch.int32, device=device)
        self.attn_cnt = torch.zeros(B * H * 2, **i32)
        self.attn_idx = torch.zeros(B * H * 2 * T, **i32)
        self.exp_cnt = torch.zeros(E + 1, **i32)
        self.exp_off = torch.zeros(E + 1, **i32)
        self.exp_rows = torch.zeros(max(B * T * k, 1), **i32)
        self.struct = Compaction(*(t.data_ptr() for t in (
            self.attn_cnt, self.attn_idx, self.exp_cnt, self.exp_off, self.exp_rows)))
