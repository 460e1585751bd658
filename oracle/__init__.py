"""CPU oracle for the verifier scoring pass (VideoSpeculateRAG, Section 3.1,
Eq. 6-7), the two-stage verification (Section 3.2, Eq. 11-15), the
multimodal retrieval stage (Section 3.1, Eq. 1-3) and the parallel draft
generation (Section 3.1, Eq. 5; Section 3.2, Eq. 8-10).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by the
benchmark's CPU-baseline leg. The product path never imports, calls or links
anything here, and nothing here imports the product package.
"""
from .decoder import (apply_rope, causal_attention, decoder_layer, embed_prefix,
                      forward_hidden, rms_norm, rope_angles, score_bruteforce,
                      score_shared_prefix, select, silu, token_log_probs)
from . import drafting, retrieval
from .verification import (ADDITION, INVERT, TWO_STAGE, branch_last_hidden, entity_alignment,
                           reliability, reliability_from_log_probs, select_final,
                           yes_no_log_probs)

__all__ = ["apply_rope", "causal_attention", "decoder_layer", "embed_prefix",
           "forward_hidden", "rms_norm", "rope_angles", "score_bruteforce",
           "score_shared_prefix", "select", "silu", "token_log_probs", "ADDITION", "INVERT",
           "TWO_STAGE", "branch_last_hidden", "entity_alignment", "reliability",
           "reliability_from_log_probs", "select_final", "yes_no_log_probs", "retrieval", "drafting"]
