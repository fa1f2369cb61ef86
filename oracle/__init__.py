"""fp64 CPU oracles for ring-chunked attention and the multi-fidelity tokenizer -- TEST
INFRASTRUCTURE ONLY.

Only the tests, the smoke check of the graft entry point and the benchmark's CPU-baseline leg may
import this package.  The HIP product path never does, and the two share no code.
"""

from .attention_fp64 import (  # noqa: F401
    attention,
    attention_bwd,
    attention_chunked,
    attention_partials,
    chunk_bounds,
    head_attention,
    head_attention_bwd,
    head_bwd_preprocess,
    head_partials,
    head_scores,
    lse_merge,
)
from .tokenizer_fp64 import (  # noqa: F401
    crop,
    gaussian_filter,
    gaussian_weights,
    mode_tokens,
    patchify,
    tt_tokenize,
)
