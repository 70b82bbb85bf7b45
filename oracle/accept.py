"""Oracle for speculative acceptance (Sec. 3.1, Sec. 3.3; greedy: Sec. 4.2).

Test infrastructure only (see the package docstring).

The paper verifies the K drafted tokens left to right with the token-wise
acceptance-rejection rule of speculative sampling: the acceptance
probability of drafted token x at position i is the ratio of its target
probability p_i(x) to its draft probability q_i(x); the first rejected
position and everything after it is discarded and that position is re-drawn
from the residual distribution built from p and q, i.e. the normalised
positive part of p_i - q_i (the rule of Leviathan et al., which the paper
cites).  Temperature 0 is greedy decoding: a drafted token is kept while it
equals the target's most likely token.

Because the device must reproduce this bit for bit, the arithmetic is fixed
exactly here.  Every step is integer arithmetic, an exact float64 product
and comparison, or one IEEE float32 subtraction, so the result does not
depend on summation order.

Readings (the paper does not spell these out):
* Accept position i iff  u_i * q_i(x_i) < p_i(x_i), evaluated in float64.
  Both factors carry at most 24 significant bits, so the product is exact
  and this is the exact test u_i < p/q, which equals u_i < min(1, p/q) for
  u_i in [0, 1).  q_i(x_i) = 0 accepts iff p_i(x_i) > 0.
* A drafted id outside [0, V) is never accepted (it cannot match a target
  token); the rows stay in bounds.
* Uniforms: u has k+1 entries per sequence; u_0..u_{k-1} drive the k
  acceptance tests and u_k drives the single final draw.  The final draw
  uses a = floor(u_k * 2^24), clamped to [0, 2^24 - 1].
* After n accepted drafts the output is draft[0..n-1] followed by one more
  token: from the residual of row n when n < k, or from the target row
  p_k (the "bonus" token) when every draft is accepted.  The output always
  holds n + 1 tokens; unused slots are -1.
* Residual weights in fixed point: r_v = max(0, p_n(v) - q_n(v)) in float32
  (round to nearest even), R_v = floor(r_v * 2^40) as an unsigned integer;
  r is clamped to [0, 1] (only invalid inputs reach the clamp).
  Values below 2^-40 weigh nothing, so flushing denormals cannot change the
  result.  S = sum_v R_v is exact for probabilities in [0, 1] and V <= 2^18.
* Inverse CDF: T = floor(a * S / 2^24); the token is the smallest j whose
  inclusive prefix sum of R exceeds T.  Such j exists and has R_j > 0.
* Degenerate residual (S = 0, possible only for unnormalised inputs): use
  R_v = floor(p_n(v) * 2^40) instead; if that is zero too, take argmax p_n.
* p and q are used as given (no renormalisation); temperature is applied by
  the caller when it builds p and q.
* Greedy: g_i = argmax_v p_i(v) comparing float32 values, lowest index on
  ties; n is the length of the longest prefix with draft[i] == g_i; the
  extra token is g_n.  q and u are not read.
"""

import numpy as np

ACCEPT_GREEDY = 0
ACCEPT_SAMPLED = 1

FIXED_POINT_BITS = 40   # residual weights are floor(r * 2^40)
UNIFORM_BITS = 24       # the final draw uses a 24-bit integer uniform


def accept_flags(p_x, q_x, u):
    """Exact acceptance tests u * q(x) < p(x) on float32 inputs (float64 math)."""
    p_x = np.asarray(p_x, dtype=np.float32).astype(np.float64)
    q_x = np.asarray(q_x, dtype=np.float32).astype(np.float64)
    u = np.asarray(u, dtype=np.float32).astype(np.float64)
    return u * q_x < p_x


def residual_weights(p_row, q_row=None):
    """Fixed-point weights R_v = floor(max(0, p_v - q_v) * 2^40) as uint64.

    The subtraction is one float32 operation (numpy float32 arithmetic is
    IEEE round-to-nearest-even); scaling by a power of two and flooring are
    exact in float64.  With ``q_row`` None the weights are floor(p_v * 2^40).
    """
    p_row = np.asarray(p_row, dtype=np.float32)
    if q_row is None:
        r = p_row
    else:
        r = np.maximum(np.float32(0.0), p_row - np.asarray(q_row, dtype=np.float32))
    # probabilities lie in [0, 1]; values outside (invalid input) are clamped
    r = np.minimum(np.maximum(r, np.float32(0.0)), np.float32(1.0))
    scaled = np.floor(r.astype(np.float64) * float(2 ** FIXED_POINT_BITS))
    return scaled.astype(np.uint64)


def uniform_to_int(u):
    """a = floor(u * 2^24) clamped to [0, 2^24 - 1] (exact for float32 u)."""
    u = np.asarray(u, dtype=np.float32).astype(np.float64)
    a = np.floor(u * float(2 ** UNIFORM_BITS))
    a = np.clip(a, 0.0, float(2 ** UNIFORM_BITS - 1))
    return a.astype(np.uint64)


def fixed_point_sample(R, a):
    """Inverse-CDF draw from integer weights R with 24-bit integer uniforms a.

    R: uint64 [V] with S = sum(R) > 0 and S < 2^58.  a: integer(s) in
    [0, 2^24).  Returns, for each a, the smallest j with
    sum_{v <= j} R_v > T where T = floor(a * S / 2^24).

    a * S can reach 2^82, so T is formed from S = S_hi * 2^24 + S_lo as
    a * S_hi + floor(a * S_lo / 2^24), every term exact in uint64.
    """
    R = np.asarray(R, dtype=np.uint64)
    S = int(np.sum(R, dtype=np.uint64))
    if S <= 0:
        raise ValueError("weights sum to zero")
    if S >= 2 ** 58:
        raise ValueError("weight sum too large for exact fixed point")
    a_arr = np.atleast_1d(np.asarray(a, dtype=np.uint64))
    s_hi = np.uint64(S >> UNIFORM_BITS)
    s_lo = np.uint64(S & (2 ** UNIFORM_BITS - 1))
    T = a_arr * s_hi + ((a_arr * s_lo) >> np.uint64(UNIFORM_BITS))
    cum = np.cumsum(R, dtype=np.uint64)
    tok = np.searchsorted(cum, T, side="right")
    if np.isscalar(a) or np.ndim(a) == 0:
        return int(tok[0])
    return tok.astype(np.int64)


def _argmax_lowest(row):
    """Index of the largest float32 value, lowest index on ties."""
    return int(np.argmax(np.asarray(row, dtype=np.float32)))


def spec_accept_one(p, q, draft, u, mode):
    """Acceptance for one sequence.

    p: [k+1, V] target probabilities; q: [k, V] draft probabilities (unused in
    greedy mode); draft: [k] drafted ids; u: [k+1] uniforms in [0, 1)
    (unused in greedy mode).  Returns (n_accepted, tokens[k+1]) where the
    first n_accepted + 1 tokens are valid and the rest are -1.
    """
    p = np.asarray(p, dtype=np.float32)
    kp1, V = p.shape
    k = kp1 - 1
    draft = [int(x) for x in np.asarray(draft).reshape(-1).tolist()]
    if len(draft) != k:
        raise ValueError("draft must hold k ids")
    tokens = [-1] * (k + 1)

    if mode == ACCEPT_GREEDY:
        n = 0
        g = _argmax_lowest(p[0])
        while n < k and draft[n] == g:
            tokens[n] = draft[n]
            n += 1
            g = _argmax_lowest(p[n])
        tokens[n] = g
        return n, tokens

    if mode != ACCEPT_SAMPLED:
        raise ValueError("unknown acceptance mode")
    q = np.asarray(q, dtype=np.float32)
    u = np.asarray(u, dtype=np.float32).reshape(-1)
    n = 0
    while n < k:
        x = draft[n]
        if not (0 <= x < V):
            break
        if not bool(accept_flags(p[n, x], q[n, x], u[n])):
            break
        tokens[n] = x
        n += 1

    if n < k:
        R = residual_weights(p[n], q[n])
    else:
        R = residual_weights(p[k])
    if int(np.sum(R, dtype=np.uint64)) == 0:
        R = residual_weights(p[n])
    if int(np.sum(R, dtype=np.uint64)) == 0:
        tokens[n] = _argmax_lowest(p[n])
    else:
        tokens[n] = fixed_point_sample(R, uniform_to_int(u[k]))
    return n, tokens


def spec_accept(p, q, draft, u, mode):
    """Batched acceptance: p [B, k+1, V], q [B, k, V], draft [B, k], u [B, k+1].

    Returns (n_accepted [B] int32, tokens [B, k+1] int32).
    """
    p = np.asarray(p, dtype=np.float32)
    B, kp1, V = p.shape
    k = kp1 - 1
    n_out = np.zeros(B, dtype=np.int32)
    tok_out = np.full((B, k + 1), -1, dtype=np.int32)
    for b in range(B):
        qb = None if q is None else np.asarray(q)[b]
        ub = None if u is None else np.asarray(u)[b]
        n, toks = spec_accept_one(p[b], qb, np.asarray(draft)[b], ub, mode)
        n_out[b] = n
        tok_out[b] = toks
    return n_out, tok_out
