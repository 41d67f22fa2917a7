"""Shared helpers of the GPU parity tests: tolerance checks (bf16: allclose
with atol 2e-3, rtol 1e-2; fp32: |d| <= 1e-5 (|ref| + rms(ref))) and input
set-up.  Inputs come from the seeded generator only."""
from __future__ import annotations

import numpy as np
import torch

import gen
import oracle
from oracle.ties import enforce_margins

BF16_ATOL, BF16_RTOL = 2e-3, 1e-2
F32_RTOL = 1e-5


def npy(t):
    return t.detach().float().cpu().numpy() if t.dtype in (torch.bfloat16, torch.float16) \
        else t.detach().cpu().numpy()


def assert_close(gpu, ref, act, name=""):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (name, gpu.shape, ref.shape)
    err = np.abs(gpu - ref)
    if act == "bf16":
        bound = BF16_ATOL + BF16_RTOL * np.abs(ref)
    else:
        rms = np.sqrt(np.mean(ref ** 2)) if ref.size else 0.0
        bound = F32_RTOL * (np.abs(ref) + rms)
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(
            f"{name}: {int(bad.sum())}/{bad.size} outside tolerance ({act}); worst at {i}: "
            f"gpu {gpu[i]!r} ref {ref[i]!r}; max abs err {err.max():.3e}")
    return float(err.max()) if err.size else 0.0


def layer(name, seed=None, moe=True, act=None):
    """Generator layer with routing kept off ties (decisions well defined)."""
    L = gen.make_layer(name, seed, with_moe=moe, act=act)
    L["resampled"] = enforce_margins(L)
    return L


def torch_act(act):
    return torch.bfloat16 if act == "bf16" else torch.float32


def shape_of(name, **over):
    s = dict(gen.CONFIGS[name])
    s.update(over)
    return s
