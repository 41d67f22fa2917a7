"""A decode step through a stack of routed layers.

TEST INFRASTRUCTURE (part of the CPU oracle): only tests use it.  It shares
no code with the GPU path.

Paper anchors: Sec. 3.3 lists the previous layer's decisions among the
causal side features psi of a layer's controller; Sec. 3.8 runs inference as
one left-to-right pass with per-token decisions taken layer by layer.

Reading (R33 in the design notes): layer l > 0 takes the caller's features
with the last four replaced by layer l - 1's decisions of the same token:
the fraction of its heads in full mode, the fraction in local mode, its
width index / 3 and its fraction of real (non-null) expert slots.  Layer
l's output (held in the activation dtype) is layer l + 1's input.
"""
import numpy as np

from .layer import MODE_FULL, MODE_LOCAL, layer_decode, to_native


def psi_next(psi, mode, bit, eidx):
    """Side features of the next layer from this layer's decisions, as the
    fp32 values a layer's side-feature input holds (each quotient rounded
    once)."""
    out = np.array(psi, np.float64, copy=True)
    H, k = mode.shape[1], eidx.shape[1]
    out[:, -4] = (np.asarray(mode) == MODE_FULL).sum(axis=1) / H
    out[:, -3] = (np.asarray(mode) == MODE_LOCAL).sum(axis=1) / H
    out[:, -2] = np.asarray(bit, np.float64) / 3.0
    out[:, -1] = (np.asarray(eidx) != 0).sum(axis=1) / k
    return out.astype(np.float32).astype(np.float64)


def stack_decode(Ls, seqs=None, x_in=None, kv_in=None, o_in=None, xt_in=None):
    """One decode step through the layers ``Ls`` (dicts as for layer_decode;
    layer 0's x and psi are the stack's inputs).

    Forced evaluation, per layer l (the comparison protocol of layer_decode):
    ``x_in[l]`` [B, d] replaces layer l's input (l >= 1) by another
    computation's output of layer l - 1; ``kv_in[l]``, ``o_in[l]``,
    ``xt_in[l]`` as layer_decode's.  Returns one layer_decode result per layer
    (its ``psi`` added)."""
    psi0 = np.asarray(Ls[0]["psi"], np.float64)
    psi = psi0
    x = Ls[0]["x"]
    act = Ls[0]["cfg"]["act"]
    out = []
    for l, L in enumerate(Ls):
        if l > 0:
            x = x_in[l] if x_in is not None and l in x_in else x
        Ll = dict(L, x=np.asarray(x), psi=psi)
        f = lambda d: None if d is None or l not in d else d[l]
        r = layer_decode(Ll, seqs, kv_in=f(kv_in), o_in=f(o_in), xt_in=f(xt_in))
        r["psi"] = psi
        out.append(r)
        psi = psi_next(psi0, r["mode"], r["bit"], r["eidx"])
        # the next input: this layer's output where computed (the compared
        # rows), held in the activation dtype
        xn = np.array(Ll["x"], np.float64, copy=True)
        xn[r["rows"]] = to_native(r["xout"], act)
        x = xn
    return out
