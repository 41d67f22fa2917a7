"""Upload a layer's weights/inputs to device tensors and fill the ABI structs.

Marshalling only: arrays in, torch tensors + ctypes structs out.
"""
from __future__ import annotations

import numpy as np
import torch

from . import (BF16, Cfg, DenseW, MoeW, RouterW, make_cfg)


def cfg_from(shape: dict, act: str | None = None) -> Cfg:
    """Build a triroute_cfg from a workload shape dict (d, H, Hkv, dh, w, E, k,
    d_ff, G, act; optional attn_groups)."""
    return make_cfg(shape["d"], shape["H"], shape["Hkv"], shape["dh"], shape["w"],
                    shape["E"], shape["k"], shape["d_ff"], shape["G"], act or shape["act"],
                    attn_groups=shape.get("attn_groups", 0) or 0)


def to_dev(a, dtype, device="cuda"):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device=device, dtype=dtype).contiguous()


class DeviceLayer:
    """Device copies of one layer's weights (and optionally its inputs)."""

    @staticmethod
    def cfg_only(L: dict) -> Cfg:
        return cfg_from(L["cfg"])

    def __init__(self, L: dict, device="cuda", moe: bool = True):
        cfg = L["cfg"]
        self.cfg = cfg_from(cfg)
        self.act = torch.bfloat16 if self.cfg.act == BF16 else torch.float32
        f32 = torch.float32
        self.t = {}
        for name in ("g1", "W1", "b1", "W2", "b2", "gr", "Wa", "ca", "We", "ce", "Wb", "cb"):
            self.t[name] = to_dev(np.asarray(L[name], np.float32), f32, device)
        self.rw = RouterW(*(self.t[n].data_ptr() for n in (
            "g1", "W1", "b1", "W2", "b2", "gr", "Wa", "ca", "We", "ce", "Wb", "cb")))
        # Wq, Wk, Wv back to back in one buffer: the many-token QKV kernel
        # addresses all three from one base (within 4 GB of it)
        qkv = [to_dev(L[n], self.act, device) for n in ("Wq", "Wk", "Wv")]
        flat = torch.empty(sum(w.numel() for w in qkv), dtype=self.act, device=device)
        off = 0
        for name, w in zip(("Wq", "Wk", "Wv"), qkv):
            self.t[name] = flat[off:off + w.numel()].view(w.shape)
            self.t[name].copy_(w)
            off += w.numel()
        del qkv
        for name in ("Wo", "g2"):
            self.t[name] = to_dev(L[name], self.act, device)
        self.dw = DenseW(*(self.t[n].data_ptr() for n in ("Wq", "Wk", "Wv", "Wo", "g2")))
        self.mw = None
        if moe and "Wg" in L:
            for name in ("Wg", "Wu", "Wd"):
                self.t[name] = to_dev(L[name], self.act, device)
            self.mw = MoeW(*(self.t[n].data_ptr() for n in ("Wg", "Wu", "Wd")))
        self.x = to_dev(L["x"], self.act, device)
        self.psi = to_dev(L["psi"], f32, device)
