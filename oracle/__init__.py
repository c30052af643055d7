"""CPU oracle for the NiuTrans deep-encoder / shallow-decoder translation path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package's smoke check and the
benchmark's CPU-baseline leg may import this package.  The product path (the HIP
library and its Python binding) never imports, calls or links anything here, and
this package imports nothing from the product path: the two share only the seeded
input generators in ``synth``.

The oracle is plain and slow on purpose: NumPy, fp64 by default (fp32 for the timed
CPU baseline), one sentence at a time, no padding, no batching.  Where the paper
fixes a definition (DLCL, Sec. 2.1 Eq. 1-2; caching, Sec. 4.1; greedy search,
Sec. 4.4; the faster beam search stop rule, Sec. 4.1) the code writes it out
directly; the readings of points the paper leaves open are listed in the module
docstrings of ``oracle.model`` and ``oracle.search``.

Parity status: every function is pinned by CPU tests (tests/test_oracle_*.py)
against library routines (torch CPU fp64 Transformer layers), closed forms,
invariants and brute force.  Absolute logits of the full model on random weights
have no value printed in the paper and are pinned only through those checks.
"""
from .model import (  # noqa: F401
    OracleModel, layer_norm, positional_encoding, softmax, logsumexp, attention,
    round_weights, param_count_formula, e4m3_round, quantize_fp8_columns,
)
from .search import (  # noqa: F401
    greedy_search, beam_search, length_penalty, Hypothesis, translate, brute_force_best,
)
