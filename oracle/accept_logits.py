"""Acceptance from logits: temperature softmax and counter-based uniforms.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The acceptance rule itself is ``oracle.accept.spec_accept`` (Sec. 3.1,
Sec. 3.3).  This module states the two steps in front of it when the target
and the draft hand over logits instead of probabilities:

* the temperature softmax that turns logits into the distributions P and P'
  of Algorithm 1 (Sec. 4.2 fixes the temperatures used), in float64 and then
  rounded to float32, the precision the rule takes its probabilities in;
* the uniforms of the tests and of the final draw, from the counter-based
  generator Philox-4x64-10 of Salmon, Moraes, Dror and Shaw ("Parallel random
  numbers: as easy as 1, 2, 3", SC'11), so that any processor can produce the
  uniform of (sequence, position) without shared state.

Readings (the paper specifies no generator):

* Philox-4x64 with 10 rounds, key (seed, 0), counter (j, b, offset, 0) for
  sequence b and block j of four outputs; uniform i of sequence b is word
  i mod 4 of block j = i div 4, and u = (word >> 40) * 2^-24, a multiple of
  2^-24 in [0, 1) as the acceptance rule expects.
* Greedy mode takes g_i = argmax_v z_i(v) of the target logits (lowest index
  on ties); the temperature plays no part (it is the tau -> 0 limit).
"""

import numpy as np

from .accept import ACCEPT_GREEDY, ACCEPT_SAMPLED, spec_accept
from .lm_head import softmax_temperature

MASK64 = (1 << 64) - 1
# round multipliers and the Weyl increments of the key (Salmon et al., the
# 4x64 variant)
PHILOX_M = (0xD2E7470EE14C6C93, 0xCA5A826395121157)
PHILOX_W = (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)


def philox4x64(counter, key, rounds=10):
    """One Philox-4x64 block: four 64-bit words from a 4-word counter and a
    2-word key (Python integers).  Each round multiplies words 0 and 2 by the
    round constants (128-bit products split into high and low halves), mixes
    the high halves with words 1, 3 and the key, and bumps the key by the Weyl
    increments."""
    c = [int(x) & MASK64 for x in counter]
    k = [int(x) & MASK64 for x in key]
    for _ in range(rounds):
        p0 = PHILOX_M[0] * c[0]
        p1 = PHILOX_M[1] * c[2]
        hi0, lo0 = p0 >> 64, p0 & MASK64
        hi1, lo1 = p1 >> 64, p1 & MASK64
        c = [hi1 ^ c[1] ^ k[0], lo1, hi0 ^ c[3] ^ k[1], lo0]
        k = [(k[0] + PHILOX_W[0]) & MASK64, (k[1] + PHILOX_W[1]) & MASK64]
    return c


def philox_uniforms(seed, offset, B, n):
    """u [B, n] float32: uniform i of sequence b as stated in the readings."""
    u = np.empty((B, n), dtype=np.float32)
    for b in range(B):
        for j in range((n + 3) // 4):
            words = philox4x64((j, b, offset, 0), (seed, 0))
            for w in range(4):
                i = 4 * j + w
                if i < n:
                    u[b, i] = np.float32((words[w] >> 40) * 2.0 ** -24)
    return u


def spec_accept_logits(target_logits, draft_logits, draft, seed, offset, tau, mode):
    """Acceptance from logits.

    target_logits [B, k+1, V], draft_logits [B, k, V] (any float dtype; used
    as float64), draft [B, k]; returns (n_accepted [B], tokens [B, k+1]) of
    ``spec_accept`` applied to p = softmax(z / tau), q = softmax(z' / tau)
    and the Philox uniforms (sampled), or to the target logits' argmax
    (greedy).
    """
    z = np.asarray(target_logits, dtype=np.float64)
    B, kp1, _ = z.shape
    k = kp1 - 1
    if mode == ACCEPT_GREEDY:
        # argmax of the logits, lowest index on ties: the rule's greedy step
        # compares float32 values, and logits of float32 or bf16 inputs are
        # float32 values exactly
        return spec_accept(z.astype(np.float32), None, draft, None, ACCEPT_GREEDY)
    if not tau > 0:
        raise ValueError("sampled acceptance needs a temperature > 0")
    p = softmax_temperature(z, tau)
    q = softmax_temperature(np.asarray(draft_logits, dtype=np.float64), tau)
    u = philox_uniforms(seed, offset, B, k + 1)
    return spec_accept(p, q, draft, u, ACCEPT_SAMPLED)
