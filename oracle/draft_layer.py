"""Oracle for one step of the draft's semi-autoregressive layer (Sec. 3.1;
Sec. 3.3; Algorithm 1 of Appendix B; the draft size of Sec. 4.4).

Test infrastructure only (see the package docstring).

The draft builds its textual input by a fully connected map of the
concatenated target feature and token embedding (following EAGLE, Sec. 3.1
and Algorithm 1), joins it to the compressed visual features, and runs one
transformer layer with 32 heads (the draft size the paper keeps, Sec. 4.4)
whose outputs at K placeholder positions are the hidden states of the next
K drafts, all in one pass (Sec. 3.3).  This module states one such pass for
the rows that are new in a drafting round, over the draft's cached context.

Readings (the paper names the parts, not their formulas):
* The layer is a pre-norm decoder layer of the target family (the EAGLE
  draft): x1 = x0 + Attn(RMSNorm(x0)) Wo^T, out = x1 + Down(SwiGLU(
  RMSNorm(x1))), with RMSNorm(x) = x / sqrt(mean(x^2) + eps) * w,
  SwiGLU(h) = silu(h Wg^T) * (h Wu^T), silu(z) = z / (1 + e^-z), and no
  biases except the fully connected map's.
* x0 = FC(concat(F_T, E)) = [F_T, E] W_fc^T + b_fc for every new row; a
  placeholder row carries the caller's input in the same slot (in the
  synthetic workloads a zero feature and a learned placeholder embedding).
* The draft's context (compressed visual features and earlier text) sits in
  a contiguous draft KV cache [B, Lmax, Hkv, D] of post-RoPE keys; each
  step appends the keys and values of its r new rows at positions
  pos[b] .. pos[b] + r - 1 and attends over positions 0 .. pos[b] + r - 1,
  causal inside the new rows (row j sees keys up to pos[b] + j), with
  scale 1 / sqrt(D) and grouped-query heads (query head h reads KV head
  h // (Hq / Hkv)).
* Rotary embedding with the half-split pairing: for i < D/2 the pair
  (x_i, x_{i + D/2}) is rotated by the angle p * theta^(-2i/D) at absolute
  position p.
* The fused projection weight Wqkv stacks the Hq query heads, then the Hkv
  key heads, then the Hkv value heads, each D rows; Wgu stacks the gate
  rows over the up rows.
"""

import numpy as np

from .verify import verify_attention


def rms_norm(x, w, eps):
    """x / sqrt(mean(x^2) + eps) * w over the last axis, in float64."""
    x = np.asarray(x, dtype=np.float64)
    r = np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x / r * np.asarray(w, dtype=np.float64)


def rope(x, positions, theta):
    """Rotary embedding of x [..., n, D] at positions [..., n] (half-split
    pairs, angle p * theta^(-2i/D) for pair i)."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    i = np.arange(half, dtype=np.float64)
    freq = np.power(float(theta), -2.0 * i / D)
    ang = np.asarray(positions, dtype=np.float64)[..., None] * freq
    cos, sin = np.cos(ang), np.sin(ang)
    if x.ndim == ang.ndim + 1:                 # x carries a heads axis before D
        cos, sin = cos[..., None, :], sin[..., None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1)


def linear(x, w, bias=None, residual=None):
    """x W^T (+ bias) (+ residual) in float64; x [R, K], W [N, K]."""
    y = np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64).T
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64)
    if residual is not None:
        y = y + np.asarray(residual, dtype=np.float64)
    return y


def silu(z):
    z = np.asarray(z, dtype=np.float64)
    return z / (1.0 + np.exp(-z))


def swiglu(gu):
    """silu(g) * u for gu = [g, u] along the last axis (gate half first)."""
    gu = np.asarray(gu, dtype=np.float64)
    I = gu.shape[-1] // 2
    return silu(gu[..., :I]) * gu[..., I:]


def semi_ar_layer(u, weights, k_cache, v_cache, pos, hq, hkv, eps, theta):
    """One draft step over the new rows.

    u [B, r, 2d]: concat(F_T, E) of the r new rows of each sequence (the
    last K of them placeholders).  weights: dict with fc_w [d, 2d], fc_b [d],
    ln1 [d], wqkv [(hq + 2 hkv) D, d], wo [d, hq D], ln2 [d], wgu [2I, d],
    wdown [d, I].  k_cache, v_cache [B, Lmax, hkv, D] hold the context at
    positions 0 .. pos[b] - 1.  Returns (out [B, r, d], k_cache', v_cache')
    with the new rows' keys (post-RoPE) and values written at positions
    pos[b] .. pos[b] + r - 1.
    """
    u = np.asarray(u, dtype=np.float64)
    B, r, _ = u.shape
    W = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
    d = W["fc_w"].shape[0]
    D = d // hq
    kc = np.array(k_cache, dtype=np.float64, copy=True)
    vc = np.array(v_cache, dtype=np.float64, copy=True)
    pos = np.asarray(pos, dtype=np.int64)

    x0 = linear(u.reshape(B * r, -1), W["fc_w"], W["fc_b"])
    qkv = linear(rms_norm(x0, W["ln1"], eps), W["wqkv"]).reshape(B, r, hq + 2 * hkv, D)
    positions = pos[:, None] + np.arange(r)[None, :]
    q = rope(qkv[:, :, :hq], positions, theta)
    k = rope(qkv[:, :, hq:hq + hkv], positions, theta)
    v = qkv[:, :, hq + hkv:]
    for b in range(B):
        kc[b, pos[b]:pos[b] + r] = k[b]
        vc[b, pos[b]:pos[b] + r] = v[b]
    attn, _ = verify_attention(q, kc, vc, (pos + r).astype(np.int64), 1.0 / np.sqrt(D))
    x1 = linear(attn.reshape(B * r, hq * D), W["wo"], residual=x0)
    out = linear(swiglu(linear(rms_norm(x1, W["ln2"], eps), W["wgu"])), W["wdown"], residual=x1)
    return out.reshape(B, r, d), kc, vc
