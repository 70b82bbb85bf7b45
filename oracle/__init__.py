"""Plain CPU oracle for the SpecFLASH draft-verify hot path (arXiv 2505.12728).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links this package: only the test suite, the smoke check and the CPU-baseline
leg of the benchmark do.  It shares no code with the HIP library and imports
nothing from it.

Every function is a direct, unblocked, float64 statement of what the paper
defines (or, for acceptance, of the step-by-step rule the paper cites), so a
reader can check it against the paper by eye:

* ``latent_compress``  -- the visual-token compressor, Sec. 3.2, Eq. 3
  (also Algorithm 1, Appendix B); ``latent_compress_q8`` the same on the int8
  draft's inputs (quantised drafts, Appendix A).
* ``verify_attention`` -- attention of the K drafted positions over the
  target's KV cache during the single parallel verification pass, Sec. 3.1.
* ``spec_accept``      -- token-wise acceptance / rejection with residual
  resampling (Sec. 3.1, Sec. 3.3), and greedy verification for temperature 0
  (Sec. 4.2).
* ``lm_head_probs`` / ``sample_tokens`` -- the LM head's temperature softmax
  over the vocabulary and categorical sampling of the drafts (Sec. 3.1,
  Sec. 3.3, Algorithm 1).
* ``spec_accept_logits`` / ``philox_uniforms`` -- acceptance from logits: the
  temperature softmax in front of the rule and counter-based uniforms
  (Philox-4x64-10, Salmon et al., SC'11).
* ``semi_ar_layer`` (with ``rms_norm``, ``rope``, ``linear``, ``swiglu``) --
  one step of the draft's semi-autoregressive layer over its cached context:
  the fully connected fusion of feature and embedding, then one pre-norm
  decoder layer whose placeholder rows give the next K draft states
  (Sec. 3.1, Sec. 3.3, Algorithm 1, Sec. 4.3); ``semi_ar_draft`` runs K
  drafts in K / k' passes of k' (the group size of the paper's ablation).

Readings of points the paper leaves open are stated in each module.  No
function here is "parity unpinned": every one is checked in
``tests/test_oracle_pins.py`` against closed forms, invariants, exact
enumeration or brute force.
"""

from .compress import latent_compress, softmax_rows, avg_pool_compress, latent_compress_q8, dequantize_pow2_rows
from .verify import verify_attention, gather_paged, merge_partials
from .lm_head import lm_head_logits, softmax_temperature, lm_head_probs, sample_tokens
from .accept_logits import philox4x64, philox_uniforms, spec_accept_logits
from .draft_layer import (rms_norm, rope, linear, silu, swiglu, semi_ar_layer, semi_ar_draft, bf16_round,
                          dequantize_rows, linear_q8, semi_ar_layer_q8)
from .accept import (
    spec_accept,
    spec_accept_one,
    accept_flags,
    residual_weights,
    fixed_point_sample,
    ACCEPT_GREEDY,
    ACCEPT_SAMPLED,
    FIXED_POINT_BITS,
    UNIFORM_BITS,
)

__all__ = [
    "latent_compress",
    "avg_pool_compress",
    "latent_compress_q8",
    "dequantize_pow2_rows",
    "softmax_rows",
    "verify_attention",
    "gather_paged",
    "merge_partials",
    "spec_accept",
    "spec_accept_one",
    "accept_flags",
    "residual_weights",
    "fixed_point_sample",
    "ACCEPT_GREEDY",
    "ACCEPT_SAMPLED",
    "FIXED_POINT_BITS",
    "UNIFORM_BITS",
    "lm_head_logits",
    "softmax_temperature",
    "lm_head_probs",
    "sample_tokens",
    "philox4x64",
    "philox_uniforms",
    "spec_accept_logits",
    "rms_norm",
    "rope",
    "linear",
    "silu",
    "swiglu",
    "semi_ar_layer",
    "semi_ar_draft",
    "bf16_round",
    "dequantize_rows",
    "linear_q8",
    "semi_ar_layer_q8",
]
