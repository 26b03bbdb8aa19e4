"""CPU oracle for grouped (shared-prefix) causal attention -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the package's smoke check and the bench's CPU baseline
leg may import this package. The product path (the HIP library and its
Python binding) never imports it and shares no code with it.

Every function here follows the paper's definition of the computation, the
Repeated-Prefix Forward of Section 2.1, Eq. (1): each group member's sequence
[prefix; response_i] is encoded on its own by ordinary causal attention,
Eq. (3). Lemma 1 (Section 2.2, proof in Appendix A.1) states that the
Shared-Prefix Forward gives the same outputs and gradients, so the repeated
computation is the reference the grouped kernels are checked against.

``rope`` is the step before the attention (Algorithm 1 takes rotary-encoded q
and k): the rotary embedding with the repeated-layout position ids that the
grouped layout keeps.
"""
from .attention import (  # noqa: F401
    causal_attention,
    grouped_oracle,
    key_gradients,
    query_rows,
)
from .rope import grouped_positions, inv_freq, pair_index, rope  # noqa: F401,E402
