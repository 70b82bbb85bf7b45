"""Oracle for latent-guided visual-token compression (Sec. 3.2, Eq. 3).

Test infrastructure only (see the package docstring).

Eq. 3 maps the N visual features F_V (N x d) to C compressed features with a
learnable query set (C x d):  F_hat_V = softmax(Cq . F_V^T) . F_V, where the
learned queries are the attention queries and F_V is both key and value.

Readings (the paper is silent on these points):
* Scale: Eq. 3 has no 1/sqrt(d) factor; ``scale`` multiplies the scores and
  the literal equation is scale = 1.
* Heads: with ``num_heads`` = H > 1 the width d is cut into H contiguous
  column slices of width d/H and Eq. 3 is applied to each slice on its own;
  H = 1 is Eq. 3 exactly.
* The query set is shared by every sequence of the batch; there are no
  projections or norms around Eq. 3.
* Softmax normalises over the N visual tokens (each latent's scores).
"""

import numpy as np


def softmax_rows(s):
    """Row-wise softmax of a float64 matrix: exp(s - rowmax) / rowsum.

    Subtracting the row maximum leaves the value unchanged (it cancels in the
    ratio) and keeps exp finite.  Entries equal to -inf get weight 0.
    """
    s = np.asarray(s, dtype=np.float64)
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def latent_compress(latents, feats, num_heads=1, scale=1.0, return_probs=False):
    """Eq. 3 applied per sequence and per head.

    latents: [C, d] learned queries (any real dtype; widened to float64).
    feats:   [B, N, d] visual features F_V of each sequence.
    Returns out [B, C, d] float64 with
        out[b][:, hs] = softmax(scale * latents[:, hs] @ feats[b][:, hs].T) @ feats[b][:, hs]
    for each head slice hs of width d / num_heads.  With ``return_probs`` the
    attention matrices [B, H, C, N] are returned as well.
    """
    lat = np.asarray(latents, dtype=np.float64)
    F = np.asarray(feats, dtype=np.float64)
    C, d = lat.shape
    B, N, d2 = F.shape
    if d2 != d:
        raise ValueError("latents and feats disagree on the feature width")
    if num_heads < 1 or d % num_heads != 0:
        raise ValueError("feature width must split evenly into heads")
    if N < 1:
        raise ValueError("need at least one visual token")
    dh = d // num_heads
    out = np.empty((B, C, d), dtype=np.float64)
    probs = np.empty((B, num_heads, C, N), dtype=np.float64) if return_probs else None
    for b in range(B):
        for h in range(num_heads):
            cols = slice(h * dh, (h + 1) * dh)
            query = lat[:, cols]          # the learned query set, C x dh
            kv = F[b][:, cols]            # F_V is both key and value, N x dh
            p = softmax_rows(scale * (query @ kv.T))   # C x N
            out[b][:, cols] = p @ kv
            if return_probs:
                probs[b, h] = p
    if return_probs:
        return out, probs
    return out


def avg_pool_compress(feats, C):
    """Average pooling of the N visual tokens into C features, the
    non-parametric compressor the compression ablation (Sec. 4.3) compares
    against.  Reading (the paper gives no formula): group c holds the
    contiguous tokens floor(c N / C) .. floor((c + 1) N / C) - 1 in the
    encoder's order and its feature is their mean.  feats [B, N, d];
    returns [B, C, d] float64 (1 <= C <= N)."""
    F = np.asarray(feats, dtype=np.float64)
    B, N, d = F.shape
    out = np.zeros((B, C, d), dtype=np.float64)
    for c in range(C):
        lo, hi = (c * N) // C, ((c + 1) * N) // C
        out[:, c] = F[:, lo:hi].mean(axis=1)
    return out


def dequantize_pow2_rows(q, e):
    """The values an int8 row with a power-of-two scale stands for:
    x[..., k] = q[..., k] * 2^e[...] (one exponent per row)."""
    q = np.asarray(q, dtype=np.float64)
    e = np.asarray(e, dtype=np.float64)
    return q * np.exp2(e)[..., None]


def latent_compress_q8(latents_q, latent_exp, feats_q, feat_exp, num_heads=1, scale=1.0):
    """Eq. 3 for the int8 draft's compressor (quantised drafts, Appendix A).

    Reading (the paper quantises the draft to int8 but names no scheme): the
    learned queries and the visual features are stored as int8 rows, each row
    (a latent, or a token of a sequence) with its own power-of-two scale 2^e,
    and Eq. 3 is computed on the values they stand for, q * 2^e.

    latents_q [C, d] int8, latent_exp [C] int; feats_q [B, N, d] int8,
    feat_exp [B, N] int.  Returns out [B, C, d] float64 (``latent_compress``
    of the dequantised inputs).
    """
    lat = dequantize_pow2_rows(latents_q, latent_exp)
    F = dequantize_pow2_rows(feats_q, feat_exp)
    return latent_compress(lat, F, num_heads, scale)

