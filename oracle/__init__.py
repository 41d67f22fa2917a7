"""CPU oracle for the inference forward of one TriRoute-routed layer.

TEST INFRASTRUCTURE ONLY.  Plain, slow, fp64 numpy code (the KV quantizer is
specified in fp32) written from the paper's equations.  Only ``tests/``, the
smoke check in ``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may
import it; the GPU library neither imports nor links anything here, and this
package shares no code, tables or helpers with it.

Parity pins: every function is pinned by tests in ``tests/test_oracle_*.py``
against closed forms, brute force on tiny inputs, library routines (torch) and
invariants the paper states.  Values beyond those pins (the exact numbers of a
trained layer) are "parity unpinned": the paper prints no worked example.
"""
from . import quant  # noqa: F401
from . import cost  # noqa: F401
from . import stack  # noqa: F401
from . import relax  # noqa: F401
from . import relax_grad  # noqa: F401
from .layer import (  # noqa: F401
    MODE_SKIP, MODE_LOCAL, MODE_FULL, BITS,
    rmsnorm, gelu, silu, softmax, rope,
    router_logits, decide, compact, margins,
    qkv, attention_seq, oproj, moe, layer_prefill, layer_decode,
    decode_cache_seq,
)
