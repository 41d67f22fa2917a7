"""Pins of the oracle's decode stack (Sec. 3.3 side features with the
previous layer's decisions, Sec. 3.8 layer-by-layer decisions)."""
import numpy as np

import gen
import oracle
from oracle import stack


def test_psi_next_counts_each_tokens_decisions():
    rng = np.random.default_rng(11)
    N, H, k, dpsi = 40, 12, 2, 8
    psi = rng.standard_normal((N, dpsi)).astype(np.float32)
    mode = rng.integers(0, 3, (N, H))
    bit = rng.integers(0, 4, N)
    eidx = rng.integers(0, 5, (N, k))
    out = stack.psi_next(psi, mode, bit, eidx)
    for t in range(N):
        np.testing.assert_array_equal(out[t, :dpsi - 4], psi[t, :dpsi - 4])
        full = sum(1 for h in range(H) if mode[t, h] == 2)
        local = sum(1 for h in range(H) if mode[t, h] == 1)
        real = sum(1 for j in range(k) if eidx[t, j] != 0)
        want = np.float32([full / H, local / H, bit[t] / 3, real / k])
        np.testing.assert_array_equal(out[t, dpsi - 4:], want.astype(np.float64))


def test_one_layer_stack_is_the_layer():
    Ls = gen.make_stack("410m_bf16_decode", 1)
    r = stack.stack_decode(Ls, [0, 5])[0]
    ref = oracle.layer_decode(Ls[0], [0, 5])
    np.testing.assert_array_equal(r["xout"], ref["xout"])
    np.testing.assert_array_equal(r["mode"], ref["mode"])


def test_pass_through_layer_hands_its_input_on():
    """A second layer whose heads all skip and whose gate puts all but
    e^-100 of its weight on the null expert returns its input (Sec. 3.2 (A),
    (B)), so the stack's output is the first layer's output in the
    activation dtype."""
    Ls = gen.make_stack("410m_bf16_decode", 2)
    H, E = Ls[1]["cfg"]["H"], Ls[1]["cfg"]["E"]
    Ls[1]["ca"] = np.tile(np.float32([50.0, -50.0, -50.0]), H)
    Ls[1]["ce"] = np.float32([50.0] + [-50.0] * E)
    seqs = [0, 3]
    r = stack.stack_decode(Ls, seqs)
    assert (r[1]["mode"] == oracle.MODE_SKIP).all()
    real = r[1]["eidx"][seqs] != 0
    assert (r[1]["egate"][seqs][real] < 1e-30).all()
    x1 = oracle.layer.to_native(r[0]["xout"], Ls[0]["cfg"]["act"])
    np.testing.assert_array_equal(r[1]["xout"], x1)
    # the second layer's side features carry the first layer's decisions
    want = stack.psi_next(Ls[0]["psi"], r[0]["mode"], r[0]["bit"], r[0]["eidx"])
    np.testing.assert_array_equal(r[1]["psi"], want)
