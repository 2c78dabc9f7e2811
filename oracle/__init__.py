"""Oracle for multi-head attention forward and backward on token-major activations.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct CPU
implementation in float64.  Only the tests, the smoke check and the CPU
baseline leg of the benchmark may import it; the HIP library and its Python
binding never import it, call it or fall back to it.  It shares no code with
the HIP path: no kernels, headers, helpers or constant tables.

Modules
  attention  numpy fp64 attention forward/backward, one (batch, head) at a time,
             materialising the full S x S score, probability and gradient
             matrices (the textbook definition, written out).
  brute      scalar triple loops of the same definition, for tiny inputs; used
             to cross-check ``attention``.
  proj       the projection matrix products around attention: Y = X W and its
             data and weight gradients.
  layout     the logical (b, h, s, i) -> physical offset map of a token-major
             tensor, built by the reshape-then-transpose chain itself, also
             for Q, K, V split out of one packed projection output.

Pins (tests/test_oracle.py, tests/test_oracle_cross.py, tests/test_oracle_proj.py,
tests/test_layout_oracle.py) tie each function to
something other than itself: brute force, float64 torch SDPA with autograd,
central finite differences, closed forms, invariants and the paper's own
layout examples.  Each function's docstring names the pin(s).
"""
from .attention import attn_fwd, attn_bwd, bwd_row_dot, head_probs, kv_head_of, allowed_mask  # noqa: F401
from .layout import token_major_offsets, head_split_offsets, packed_qkv_offsets  # noqa: F401
from .proj import proj_fwd, proj_bwd_data, proj_bwd_weight  # noqa: F401
