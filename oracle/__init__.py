"""CPU oracle for NaCl's encoding-phase KV-cache eviction (arXiv 2408.03675).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The GPU library never
calls it, and it shares no code with the GPU library.
"""

from .nacl_oracle import (  # noqa: F401
    SAMPLE_SOFTMAX, SAMPLE_PROPORTIONAL, SAMPLE_UNIFORM,
    proxy_scores, proxy_scores_grouped, causal_attention, protected_set, budget_split, top_k_lower_index,
    gumbel_keys, select_head, select, compact, slot_layout, evict,
)
from .philox import philox4x32_10, token_words, open_unit, seed_to_key  # noqa: F401
