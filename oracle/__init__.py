"""Plain fp64 CPU oracle for block-diffusion masked attention and for the
token log-probabilities and objectives that consume its output.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path
(the HIP library and its Python binding) never calls it.
"""
from .bd_attn_oracle import (  # noqa: F401
    block_index,
    visibility_mask,
    allowed_count,
    forward,
    backward,
    probabilities,
    sampled,
    varlen_visibility_mask,
    varlen_forward,
    varlen_backward,
    decode_forward,
)
from .lce_oracle import (  # noqa: F401
    lm_head_logprobs,
    lm_head_backward,
    masked_ce_objective,
    dipo_objective,
    lm_head_sampled,
)
