"""CPU oracle of distributed sign momentum with local steps (arXiv 2411.17866).

TEST INFRASTRUCTURE: only tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  It is independent of the HIP
library and never imports it.
"""
from .dsm_oracle import (  # noqa: F401
    PRECISIONS, SIGN_DET, SIGN_RAND_FLIP, SIGN_RAND_ZERO, PHILOX_STREAM,
    RULE_SIGN_MOMENTUM, RULE_LOOKAHEAD, RULE_SIGNED_SLOWMO, RULE_GLOBAL_ADAMW,
    beta_power, communication_round, f32, global_step, init_state,
    local_adamw_step, local_sgdm_step, local_steps, randomized_sign,
    randomized_sign_uniforms, randomized_sign_uniforms_at, sign, synchronize,
)
from .philox import philox4x32_10, philox4x32_10_scalar  # noqa: F401
