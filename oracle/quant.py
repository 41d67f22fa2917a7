"""KV-cache bit-width axis: the per-token asymmetric group quantizer.

TEST INFRASTRUCTURE (part of the CPU oracle): only tests, the smoke check and
the benchmark's CPU-baseline leg use it.  It shares no code with the GPU path.

Follows the paper's quantizer equation in Sec. 3.2 (C): for the chosen width
b, s = (max(k) - min(k)) / (2^b - 1), z = min(k), Q_b(k) = round((k - z)/s) s + z,
applied to keys and values alike; b = 16 means "keep native precision".

The paper leaves rounding, storage dtype and the arithmetic open.  This oracle
fixes them (and the GPU must reproduce them bit for bit):
  * groups of G contiguous channels within one kv-head vector of one token;
  * mn, mx, s32 = (mx - mn) / (2^b - 1) in IEEE fp32, round-to-nearest-even;
  * the stored scale and zero are fp16(s32), fp16(mn) (RNE);
  * code = 0 if fp32(s) == 0 else clamp(rint_even((x - fp32(z)) / fp32(s)), 0, 2^b-1),
    every operation in fp32;
  * dequantized value = code * s + z (evaluated here in fp64);
  * b = 16 stores the activation value verbatim.
"""
from __future__ import annotations

import numpy as np

BITS = (2, 4, 8, 16)


def quantize(x: np.ndarray, b: int, G: int):
    """Quantize the last axis of ``x`` (fp32 values) in groups of ``G``.

    Returns ``(codes uint8 [..., dh], scale fp16 [..., dh/G], zero fp16 [..., dh/G])``.
    For b = 16 returns ``(x, None, None)``.
    """
    if b == 16:
        return x, None, None
    x = np.asarray(x, dtype=np.float32)
    dh = x.shape[-1]
    assert dh % G == 0
    xg = x.reshape(x.shape[:-1] + (dh // G, G))
    mn = xg.min(axis=-1)
    mx = xg.max(axis=-1)
    levels = np.float32(2 ** b - 1)
    s32 = (mx - mn) / levels                          # fp32 subtract, fp32 divide
    s16 = s32.astype(np.float16)                      # RNE
    z16 = mn.astype(np.float16)                       # RNE
    S = s16.astype(np.float32)[..., None]
    Z = z16.astype(np.float32)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.rint((xg - Z) / S)                     # fp32 ops, ties to even
    q = np.where(S == 0, np.float32(0), np.clip(q, 0, levels))
    codes = q.astype(np.uint8).reshape(x.shape)
    return codes, s16, z16


def dequantize(codes: np.ndarray, s16: np.ndarray, z16: np.ndarray, G: int):
    """x_hat = code * s + z in fp64 (group-broadcast)."""
    c = np.asarray(codes, np.float64)
    dh = c.shape[-1]
    cg = c.reshape(c.shape[:-1] + (dh // G, G))
    out = cg * np.asarray(s16, np.float64)[..., None] + np.asarray(z16, np.float64)[..., None]
    return out.reshape(c.shape)


def roundtrip(x: np.ndarray, b: int, G: int) -> np.ndarray:
    """The value a later query reads for a token stored at width b (fp64)."""
    if b == 16:
        return np.asarray(x, np.float64)
    codes, s, z = quantize(x, b, G)
    return dequantize(codes, s, z, G)
