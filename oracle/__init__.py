"""CPU oracle for the per-operator decoder-layer forward (fp64, NumPy).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this package.  The HIP library and its
Python binding never import it and share no code with it.

Every function is the plain textbook definition of the operator the paper names
(Section 2.1's operator characterization: RMS Norm, QKV Linear and the MLP
linears, the fused SiLU-and-multiply activation, FlashAttention-style prefill
attention, decode attention over a paged KV cache) and of the operators around
them in a full layer (rotary embedding, the paged KV-cache write, the residual
add before each norm), evaluated in fp64 with no
tiling, no online softmax and no split of the key range.  See `ops` for the
per-function citations, `cost` for the algorithmic flop/byte closed forms and
`spatial` for CU shares and the interference factor of Eq. 5, `moe` for
top-k routing and the fused mixture-of-experts MLP.

Parity status: every exported function has a named pin in the CPU tests
(brute force, a hand-worked golden, a closed form or an invariant, plus planted
mistakes each pin must catch): tests/test_oracle_pins.py for `ops` and `cost`,
tests/test_oracle_moe.py for `moe`, tests/test_oracle_spatial.py for
`spatial`.  The whole-layer dataflow is pinned by a two-token layer worked by
hand (tests/golden/layer_two_tokens_hand.txt).
"""
from .ops import (  # noqa: F401
    rmsnorm, linear, silu, swiglu, softmax, attn_prefill, attn_prefill_rows,
    attn_decode, gather_paged, rope, reshape_and_cache, add_rmsnorm, decoder_layer_forward, decoder_layer_decode,
)
from . import cost  # noqa: F401
from . import spatial  # noqa: F401
from . import moe  # noqa: F401
