"""Oracle for one step of the draft's semi-autoregressive layer (Sec. 3.1;
Sec. 3.3; Algorithm 1 of Appendix B; the draft size of Sec. 4.3).

Test infrastructure only (see the package docstring).

The draft builds its textual input by a fully connected map of the
concatenated target feature and token embedding (following EAGLE, Sec. 3.1
and Algorithm 1), joins it to the compressed visual features, and runs one
transformer layer with 32 heads (the draft size the paper keeps, Sec. 4.3)
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
* The int8 draft (the quantised drafts of Appendix A name int8 without
  a scheme) is weight-only: every projection row n holds int8 values wq
  and one scale, W[n, :] = scale[n] * wq[n, :]; activations, norms and the
  FC bias stay as in the bf16 draft.
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


def bf16_round(x):
    """Round float64 values to the nearest bfloat16 value (ties to even),
    returned as float64: the precision the layer's inputs are stored in."""
    f = np.asarray(x, dtype=np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) >> 16 << 16
    return bits.astype(np.uint32).view(np.float32).astype(np.float64)


def semi_ar_draft(u0, weights, lm_w, emb, ph, k_cache, v_cache, pos, hq, hkv, eps, theta, tau,
                  uniforms, K, kp, tokens=None):
    """K drafts in K / k' passes of the semi-AR layer, k' per pass (the group
    size k' of the paper's ablation in Appendix E).

    Pass 0 runs the layer on u0 [B, r0, 2d], whose last k' rows are
    placeholders, at positions pos .. pos + r0 - 1.  After each pass the
    LM head gives the k' placeholder rows' distributions at temperature tau
    (their states rounded to bf16, the head's input precision)
    and one token is drawn per row (``sample_tokens`` with the uniforms of
    those positions, uniforms [B, K]).  The next pass takes 2k' rows: the k'
    drafted tokens, each with input concat(F', E[token]) where F' is the
    output state of the placeholder that drafted it (rounded to bf16, the
    layer's input precision), at that placeholder's position, followed by
    k' placeholder rows (input ph [2d]).  With ``tokens`` [B, K] given, those
    tokens are fed back instead of the drawn ones (the distributions are
    still those of the pass).  Returns (tokens [B, K], q [B, K, V]).
    """
    from .lm_head import lm_head_probs, sample_tokens
    u = np.asarray(u0, dtype=np.float64)
    B, r, _ = u.shape
    d = u.shape[2] // 2
    emb = np.asarray(emb, dtype=np.float64)
    ph = np.asarray(ph, dtype=np.float64)
    uniforms = np.asarray(uniforms, dtype=np.float32)
    V = np.asarray(lm_w).shape[0]
    kc, vc = k_cache, v_cache
    p = np.asarray(pos, dtype=np.int64).copy()
    out_tok = np.zeros((B, K), dtype=np.int32)
    out_q = np.zeros((B, K, V), dtype=np.float64)
    for t in range(K // kp):
        out, kc, vc = semi_ar_layer(u, weights, kc, vc, p, hq, hkv, eps, theta)
        hid = bf16_round(out[:, r - kp:]).reshape(B * kp, d)   # the head's input precision
        q = lm_head_probs(hid, lm_w, tau).reshape(B, kp, V)
        drawn = sample_tokens(q.reshape(B * kp, V).astype(np.float32),
                              uniforms[:, t * kp:(t + 1) * kp].reshape(-1)).reshape(B, kp)
        tok = drawn if tokens is None else np.asarray(tokens)[:, t * kp:(t + 1) * kp]
        out_tok[:, t * kp:(t + 1) * kp] = tok
        out_q[:, t * kp:(t + 1) * kp] = q
        text = np.concatenate([bf16_round(out[:, r - kp:]), emb[tok]], axis=-1)
        u = np.concatenate([text, np.broadcast_to(ph, (B, kp, 2 * d))], axis=1)
        p = p + (r - kp)
        r = 2 * kp
    return out_tok, out_q


def dequantize_rows(wq, scale):
    """The weight an int8 row-quantised projection stands for: W[n, k] =
    scale[n] * wq[n, k] (one scale per output row)."""
    return np.asarray(scale, dtype=np.float64)[:, None] * np.asarray(wq, dtype=np.float64)


def linear_q8(x, wq, scale, bias=None, residual=None):
    """x W^T (+ bias) (+ residual) with W = dequantize_rows(wq, scale)."""
    return linear(x, dequantize_rows(wq, scale), bias, residual)


Q8_WEIGHTS = ("fc_w", "wqkv", "wo", "wgu", "wdown")


def semi_ar_layer_q8(u, weights, k_cache, v_cache, pos, hq, hkv, eps, theta):
    """``semi_ar_layer`` of the int8 draft: weights holds, for each projection
    name in Q8_WEIGHTS, the int8 rows under that name and their scales under
    name + "_s"; the layer is the one of the dequantised weights."""
    W = {k: v for k, v in weights.items() if not k.endswith("_s")}
    for name in Q8_WEIGHTS:
        W[name] = dequantize_rows(weights[name], weights[name + "_s"])
    return semi_ar_layer(u, W, k_cache, v_cache, pos, hq, hkv, eps, theta)
