"""Oracle for the LM head that turns hidden states into token distributions
and for sampling drafts from them (Sec. 3.1; Sec. 3.3; Algorithm 1).

Test infrastructure only (see the package docstring).

The paper's LM head maps a last-layer feature to a probability distribution
over the vocabulary (Sec. 3.1).  The target's frozen LM head also projects
the draft's K hidden states into the draft distributions P'_1..P'_K, from
which the candidates are drawn, T'_i ~ Categorical(P'_i) (Sec. 3.3 and
Algorithm 1).  Generation runs at temperature tau (Sec. 4.2).

Readings (the paper gives no formula for the head):
* The head is one bias-free linear map W [V, d] followed by a softmax over
  the vocabulary of the logits divided by tau: p = softmax(h W^T / tau),
  tau > 0.  Normalisation layers before it belong to the transformer.
  Temperature 0 (greedy) takes the argmax of the logits, which the argmax of
  p at any tau > 0 reproduces, so greedy callers use any positive tau.
* Sampling uses the same exact fixed-point inverse CDF as the final draw of
  the acceptance rule (accept.py): weights floor(p_v 2^40), a 24-bit
  uniform a = floor(u 2^24), the smallest v whose inclusive prefix sum
  exceeds floor(a S / 2^24); all-zero weights fall back to argmax p.  It is
  therefore a deterministic function of the float32 probabilities and the
  uniform.
"""

import numpy as np

from .accept import residual_weights, fixed_point_sample, uniform_to_int


def lm_head_logits(hidden, weight):
    """z = hidden W^T in float64.  hidden [R, d], weight [V, d] -> [R, V]."""
    h = np.asarray(hidden, dtype=np.float64)
    w = np.asarray(weight, dtype=np.float64)
    return h @ w.T


def softmax_temperature(z, tau):
    """softmax(z / tau) along the last axis in float64 (tau > 0)."""
    if not tau > 0:
        raise ValueError("temperature must be positive")
    x = np.asarray(z, dtype=np.float64) / float(tau)
    x = x - np.max(x, axis=-1, keepdims=True)
    e = np.exp(x)
    return e / np.sum(e, axis=-1, keepdims=True)


def lm_head_probs(hidden, weight, tau):
    """Token distributions p = softmax(hidden W^T / tau), float64 [R, V]."""
    return softmax_temperature(lm_head_logits(hidden, weight), tau)


def sample_tokens(probs, u):
    """T_r ~ Categorical(probs[r]) by the exact fixed-point inverse CDF.

    probs: [R, V] float32 (used as given); u: [R] float32 uniforms in [0, 1)
    on the 2^-24 grid.  Returns int32 [R].
    """
    probs = np.asarray(probs, dtype=np.float32)
    u = np.asarray(u, dtype=np.float32).reshape(-1)
    out = np.empty(probs.shape[0], dtype=np.int32)
    for r in range(probs.shape[0]):
        weights = residual_weights(probs[r])
        if int(np.sum(weights, dtype=np.uint64)) == 0:
            out[r] = int(np.argmax(probs[r]))
        else:
            out[r] = fixed_point_sample(weights, uniform_to_int(u[r]))
    return out
