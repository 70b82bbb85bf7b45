"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, an invariant, an exact enumeration, hand-worked cases, or brute force
on tiny inputs.  They run on the CPU only.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed=0):
    return np.random.default_rng(seed)


# ================================================================ compression
# Eq. 3 (Sec. 3.2): out = softmax(scale * Cq F_V^T) F_V, per head slice.

@pytest.mark.parametrize("heads,scale", [(1, 1.0), (4, 0.5), (2, 1 / math.sqrt(8))])
def test_compress_zero_queries_is_average_pooling(heads, scale):
    # Cq = 0 makes every score equal, so each latent averages all N tokens:
    # global average pooling (the pooling compressor of the compression ablation in Sec. 4.3).
    r = rng(1)
    feats = r.standard_normal((3, 7, 16))
    out = oracle.latent_compress(np.zeros((5, 16)), feats, heads, scale)
    expect = np.broadcast_to(feats.mean(axis=1)[:, None, :], out.shape)
    np.testing.assert_allclose(out, expect, rtol=0, atol=1e-13)


def test_compress_two_token_logistic_closed_form():
    # N = 2: weights are the logistic function of the score difference.
    r = rng(2)
    f = r.standard_normal((1, 2, 6))
    c = r.standard_normal((3, 6))
    scale = 0.37
    out = oracle.latent_compress(c, f, 1, scale)
    for i in range(3):
        s0 = scale * float(np.dot(c[i], f[0, 0]))
        s1 = scale * float(np.dot(c[i], f[0, 1]))
        w0 = 1.0 / (1.0 + math.exp(s1 - s0))
        expect = w0 * f[0, 0] + (1.0 - w0) * f[0, 1]
        np.testing.assert_allclose(out[0, i], expect, rtol=0, atol=1e-13)


def test_compress_value_is_the_feature_itself():
    # One-hot limit: a query equal to lambda * (unit row j) attends to row j
    # only, and returns that row: F_V is both key and value.
    r = rng(3)
    f = r.standard_normal((1, 9, 12))
    f /= np.linalg.norm(f, axis=-1, keepdims=True)
    picks = [4, 0, 8]
    c = 400.0 * f[0, picks]
    out = oracle.latent_compress(c, f, 1, 1.0)
    np.testing.assert_allclose(out[0], f[0, picks], rtol=0, atol=1e-12)


def test_compress_token_order_does_not_matter():
    r = rng(4)
    f = r.standard_normal((2, 11, 8))
    c = r.standard_normal((4, 8))
    perm = r.permutation(11)
    a = oracle.latent_compress(c, f, 2, 0.7)
    b = oracle.latent_compress(c, f[:, perm], 2, 0.7)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_compress_single_and_repeated_token():
    r = rng(5)
    row = r.standard_normal(8)
    c = r.standard_normal((3, 8))
    one = oracle.latent_compress(c, row[None, None, :], 2, 1.0)
    np.testing.assert_allclose(one[0], np.broadcast_to(row, (3, 8)), atol=1e-15)
    many = oracle.latent_compress(c, np.broadcast_to(row, (1, 6, 8)).copy(), 2, 1.0)
    np.testing.assert_allclose(many[0], np.broadcast_to(row, (3, 8)), atol=1e-14)


def test_compress_heads_are_contiguous_slices():
    # Head 0 has zero queries (mean of its slice); head 1 has one-hot queries
    # (the picked row of its slice).  Only contiguous slices give both.
    r = rng(6)
    f = r.standard_normal((1, 5, 8))
    f[0, :, 4:] /= np.linalg.norm(f[0, :, 4:], axis=-1, keepdims=True)
    c = np.zeros((2, 8))
    c[0, 4:] = 500.0 * f[0, 3, 4:]
    c[1, 4:] = 500.0 * f[0, 1, 4:]
    out = oracle.latent_compress(c, f, 2, 1.0)
    np.testing.assert_allclose(out[0, :, :4], np.broadcast_to(f[0, :, :4].mean(0), (2, 4)), atol=1e-13)
    np.testing.assert_allclose(out[0, 0, 4:], f[0, 3, 4:], atol=1e-12)
    np.testing.assert_allclose(out[0, 1, 4:], f[0, 1, 4:], atol=1e-12)


def test_compress_probabilities_sum_to_one():
    r = rng(7)
    _, probs = oracle.latent_compress(r.standard_normal((4, 8)),
                                      r.standard_normal((2, 13, 8)) * 5, 2, 1.0,
                                      return_probs=True)
    np.testing.assert_allclose(probs.sum(-1), 1.0, rtol=0, atol=1e-12)
    assert np.all(probs >= 0)


def test_compress_brute_force_tiny():
    # Pure-Python loops over (b, head, latent, token) on a tiny case.
    r = rng(8)
    C, N, d, H, B = 3, 5, 8, 2, 2
    c = r.standard_normal((C, d))
    f = r.standard_normal((B, N, d))
    scale = 0.8
    out = oracle.latent_compress(c, f, H, scale)
    dh = d // H
    for b in range(B):
        for h in range(H):
            for i in range(C):
                s = [scale * sum(c[i, h * dh + t] * f[b, n, h * dh + t] for t in range(dh))
                     for n in range(N)]
                z = sum(math.exp(x) for x in s)
                for t in range(dh):
                    v = sum(math.exp(s[n]) / z * f[b, n, h * dh + t] for n in range(N))
                    assert abs(v - out[b, i, h * dh + t]) < 1e-12


# ============================================================== verification
# Attention of the k-token block over the cache (Sec. 3.1), causal in block.

def test_verify_single_key_returns_its_value():
    r = rng(10)
    q = r.standard_normal((1, 1, 2, 4))
    K = r.standard_normal((1, 1, 1, 4))
    V = r.standard_normal((1, 1, 1, 4))
    out, lse = oracle.verify_attention(q, K, V, [1], 0.5)
    np.testing.assert_allclose(out[0, 0], np.broadcast_to(V[0, 0, 0], (2, 4)), atol=1e-15)
    np.testing.assert_allclose(lse[0, 0], 0.5 * q[0, 0] @ K[0, 0, 0], atol=1e-15)


def test_verify_equal_keys_average_exactly_the_visible_prefix():
    # With identical keys every visible score is equal, so row j returns the
    # mean of the first L - k + j + 1 values and lse = s + log(count).
    r = rng(11)
    B, k, Hq, Hkv, D, L = 2, 3, 2, 1, 4, 9
    q = r.standard_normal((B, k, Hq, D))
    key = r.standard_normal(D)
    K = np.broadcast_to(key, (B, L, Hkv, D)).copy()
    V = r.standard_normal((B, L, Hkv, D))
    lens = [9, 5]
    out, lse = oracle.verify_attention(q, K, V, lens, 0.3)
    for b in range(B):
        for j in range(k):
            n_vis = lens[b] - k + j + 1
            for h in range(Hq):
                np.testing.assert_allclose(out[b, j, h], V[b, :n_vis, 0].mean(0), atol=1e-14)
                s = 0.3 * float(q[b, j, h] @ key)
                assert abs(lse[b, j, h] - (s + math.log(n_vis))) < 1e-13


def test_verify_two_key_logistic_closed_form():
    r = rng(12)
    q = r.standard_normal((1, 1, 1, 5))
    K = r.standard_normal((1, 2, 1, 5))
    V = r.standard_normal((1, 2, 1, 5))
    scale = 0.61
    out, lse = oracle.verify_attention(q, K, V, [2], scale)
    s0 = scale * float(q[0, 0, 0] @ K[0, 0, 0])
    s1 = scale * float(q[0, 0, 0] @ K[0, 1, 0])
    w0 = 1.0 / (1.0 + math.exp(s1 - s0))
    np.testing.assert_allclose(out[0, 0, 0], w0 * V[0, 0, 0] + (1 - w0) * V[0, 1, 0], atol=1e-14)
    assert abs(lse[0, 0, 0] - math.log(math.exp(s0) + math.exp(s1))) < 1e-13


def test_verify_gqa_heads_read_contiguous_groups():
    # Value rows of KV head c are all (c + 1): query head h must return
    # h // g + 1 whatever the scores are.
    r = rng(13)
    B, k, Hq, Hkv, D, L = 1, 2, 8, 2, 4, 6
    q = r.standard_normal((B, k, Hq, D))
    K = r.standard_normal((B, L, Hkv, D))
    V = np.zeros((B, L, Hkv, D))
    for c in range(Hkv):
        V[:, :, c, :] = c + 1.0
    out, _ = oracle.verify_attention(q, K, V, [L], 0.5)
    g = Hq // Hkv
    for h in range(Hq):
        np.testing.assert_allclose(out[0, :, h], h // g + 1.0, atol=1e-14)


def test_verify_gqa_equals_repeated_kv():
    r = rng(14)
    B, k, Hq, Hkv, D, L = 2, 3, 6, 2, 8, 10
    q = r.standard_normal((B, k, Hq, D))
    K = r.standard_normal((B, L, Hkv, D))
    V = r.standard_normal((B, L, Hkv, D))
    a, la = oracle.verify_attention(q, K, V, [10, 7], 0.4)
    Kr = np.repeat(K, Hq // Hkv, axis=2)
    Vr = np.repeat(V, Hq // Hkv, axis=2)
    b, lb = oracle.verify_attention(q, Kr, Vr, [10, 7], 0.4)
    np.testing.assert_allclose(a, b, atol=1e-14)
    np.testing.assert_allclose(la, lb, atol=1e-14)


def test_verify_block_row_is_a_single_query_decode():
    # Row j of the block equals one-query attention over the first
    # L - k + j + 1 cache entries; the last row sees the whole cache.
    r = rng(15)
    B, k, Hq, Hkv, D, L = 1, 4, 4, 2, 8, 12
    q = r.standard_normal((B, k, Hq, D))
    K = r.standard_normal((B, L, Hkv, D))
    V = r.standard_normal((B, L, Hkv, D))
    out, lse = oracle.verify_attention(q, K, V, [L], 0.25)
    for j in range(k):
        n_vis = L - k + j + 1
        o1, l1 = oracle.verify_attention(q[:, j:j + 1], K[:, :n_vis], V[:, :n_vis], [n_vis], 0.25)
        np.testing.assert_allclose(out[:, j], o1[:, 0], atol=1e-14)
        np.testing.assert_allclose(lse[:, j], l1[:, 0], atol=1e-14)


def test_verify_masked_entries_are_never_read():
    # Poisoning cache slots past kv_len (NaN) changes nothing, and changing
    # the last block entry changes only the last block row.
    r = rng(16)
    B, k, Hq, Hkv, D, Lmax = 2, 3, 2, 1, 4, 10
    q = r.standard_normal((B, k, Hq, D))
    K = r.standard_normal((B, Lmax, Hkv, D))
    V = r.standard_normal((B, Lmax, Hkv, D))
    lens = [8, 6]
    base, lb = oracle.verify_attention(q, K, V, lens, 0.5)
    Kp, Vp = K.copy(), V.copy()
    for b, L in enumerate(lens):
        Kp[b, L:] = np.nan
        Vp[b, L:] = np.nan
    pois, lp = oracle.verify_attention(q, Kp, Vp, lens, 0.5)
    np.testing.assert_array_equal(base, pois)
    np.testing.assert_array_equal(lb, lp)
    K2, V2 = K.copy(), V.copy()
    K2[0, lens[0] - 1] += 3.0
    V2[0, lens[0] - 1] -= 2.0
    changed, _ = oracle.verify_attention(q, K2, V2, lens, 0.5)
    np.testing.assert_array_equal(changed[0, :k - 1], base[0, :k - 1])
    assert np.max(np.abs(changed[0, k - 1] - base[0, k - 1])) > 1e-3


def test_verify_rows_without_keys_are_zero():
    r = rng(17)
    q = r.standard_normal((1, 4, 2, 4))
    K = r.standard_normal((1, 4, 1, 4))
    V = r.standard_normal((1, 4, 1, 4))
    out, lse = oracle.verify_attention(q, K, V, [2], 1.0)
    # kv_len 2 < k 4: rows 0 and 1 see no key, rows 2, 3 see 1 and 2 keys
    assert np.all(out[0, :2] == 0) and np.all(np.isneginf(lse[0, :2]))
    np.testing.assert_allclose(out[0, 2], np.broadcast_to(V[0, 0, 0], (2, 4)), atol=1e-15)


def test_verify_paged_equals_contiguous():
    r = rng(18)
    B, k, Hq, Hkv, D, ps = 3, 2, 4, 2, 8, 16
    lens = [40, 17, 33]
    Lmax = 48
    q = r.standard_normal((B, k, Hq, D))
    K = r.standard_normal((B, Lmax, Hkv, D))
    V = r.standard_normal((B, Lmax, Hkv, D))
    pages = [math.ceil(L / ps) for L in lens]
    n_pool = sum(pages) + 3
    perm = r.permutation(n_pool)
    table = np.zeros((B, 3), dtype=np.int32)
    kp = np.full((n_pool, Hkv, ps, D), np.nan)
    vp = np.full((n_pool, Hkv, ps, D), np.nan)
    pos = 0
    for b in range(B):
        for i in range(pages[b]):
            pg = perm[pos]
            pos += 1
            table[b, i] = pg
            for s in range(ps):
                t = i * ps + s
                if t < lens[b]:
                    kp[pg, :, s] = K[b, t]
                    vp[pg, :, s] = V[b, t]
    a, la = oracle.verify_attention(q, K, V, lens, 0.3)
    b_, lb = oracle.verify_attention(q, kp, vp, lens, 0.3, page_table=table, page_size=ps)
    np.testing.assert_array_equal(a, b_)
    np.testing.assert_array_equal(la, lb)


def test_verify_merge_of_key_partition_equals_whole():
    # The log-sum-exp merge of attention over disjoint key ranges equals
    # attention over their union; this pins lse.
    r = rng(19)
    D, L, Hq = 8, 30, 3
    q = r.standard_normal((1, 1, Hq, D))
    K = r.standard_normal((1, L, 1, D)) * 2
    V = r.standard_normal((1, L, 1, D))
    whole, lw = oracle.verify_attention(q, K, V, [L], 0.7)
    cuts = [0, 4, 5, 19, 30]
    outs, lses = [], []
    for a, b in zip(cuts[:-1], cuts[1:]):
        o, l_ = oracle.verify_attention(q, K[:, a:b], V[:, a:b], [b - a], 0.7)
        outs.append(o)
        lses.append(l_)
    o, l_ = oracle.merge_partials(np.stack(outs), np.stack(lses))
    np.testing.assert_allclose(o, whole, atol=1e-13)
    np.testing.assert_allclose(l_, lw, atol=1e-13)


def test_verify_probabilities_sum_to_one():
    r = rng(20)
    q = r.standard_normal((2, 3, 4, 8)) * 3
    K = r.standard_normal((2, 12, 2, 8))
    V = r.standard_normal((2, 12, 2, 8))
    _, _, probs = oracle.verify_attention(q, K, V, [12, 9], 0.5, return_probs=True)
    for b, L in enumerate([12, 9]):
        for j in range(3):
            np.testing.assert_allclose(probs[b][j].sum(-1), 1.0, atol=1e-12)
            assert np.all(probs[b][j][:, L - 3 + j + 1:] == 0)


def test_verify_brute_force_tiny():
    r = rng(21)
    B, k, Hq, Hkv, D, L = 2, 3, 4, 2, 4, 7
    q = r.standard_normal((B, k, Hq, D))
    K = r.standard_normal((B, L, Hkv, D))
    V = r.standard_normal((B, L, Hkv, D))
    lens = [7, 5]
    scale = 0.45
    out, lse = oracle.verify_attention(q, K, V, lens, scale)
    for b in range(B):
        for j in range(k):
            for h in range(Hq):
                c = h // (Hq // Hkv)
                ts = range(lens[b] - k + j + 1)
                s = [scale * sum(q[b, j, h, e] * K[b, t, c, e] for e in range(D)) for t in ts]
                z = sum(math.exp(x) for x in s)
                assert abs(lse[b, j, h] - math.log(z)) < 1e-12
                for e in range(D):
                    v = sum(math.exp(s[t]) / z * V[b, t, c, e] for t in ts)
                    assert abs(v - out[b, j, h, e]) < 1e-12


# ================================================================ acceptance
# Token-wise acceptance / residual resampling (Sec. 3.1, Sec. 3.3) and greedy
# verification at temperature 0 (Sec. 4.2).

def test_accept_hand_worked_cases():
    with open(os.path.join(GOLDEN, "accept_hand_cases.json")) as fh:
        cases = json.load(fh)["cases"]
    for c in cases:
        mode = oracle.ACCEPT_GREEDY if c["mode"] == "greedy" else oracle.ACCEPT_SAMPLED
        p = np.array(c["p"], dtype=np.float32)
        q = None if c["q"] is None else np.array(c["q"], dtype=np.float32)
        u = None if c["u"] is None else np.array(c["u"], dtype=np.float32)
        n, toks = oracle.spec_accept_one(p, q, c["draft"], u, mode)
        assert (n, toks) == (c["n"], c["tokens"]), c["name"]


def _random_probs(r, shape, temp=1.0):
    z = r.standard_normal(shape) * 3 / temp
    e = np.exp(z - z.max(-1, keepdims=True))
    return (e / e.sum(-1, keepdims=True)).astype(np.float32)


def test_accept_draft_equal_to_target_accepts_everything():
    r = rng(30)
    k, V = 6, 50
    for trial in range(20):
        p = _random_probs(r, (k + 1, V))
        draft = [int(r.integers(0, V)) for _ in range(k)]
        # keep drafted ids where p > 0 (float32 underflow could zero them)
        p[np.arange(k), draft] = np.maximum(p[np.arange(k), draft], 1e-6)
        u = (r.integers(0, 1 << 24, size=k + 1) * 2.0 ** -24).astype(np.float32)
        n, toks = oracle.spec_accept_one(p, p[:k], draft, u, oracle.ACCEPT_SAMPLED)
        assert n == k and toks[:k] == draft and 0 <= toks[k] < V


def test_accept_special_uniforms_and_ratios():
    p_x = np.array([0.3, 0.3, 0.0, 0.5, 1e-30], dtype=np.float32)
    q_x = np.array([0.1, 0.3, 0.2, 0.0, 0.0], dtype=np.float32)
    # u = 0 accepts iff p(x) > 0
    assert list(oracle.accept_flags(p_x, q_x, np.zeros(5, np.float32))) == [True, True, False, True, True]
    # p >= q accepts for every u < 1
    top = np.float32(1 - 2 ** -24)
    assert list(oracle.accept_flags(p_x[:2], q_x[:2], np.full(2, top))) == [True, True]
    # p = 0 rejects for every u
    assert not oracle.accept_flags(np.float32(0), np.float32(0.5), np.float32(0))


def test_accept_ratio_threshold_is_exact():
    # accept iff u < p/q exactly: on the 2^-24 grid the number of accepting
    # uniforms is ceil(2^24 * p / q) (capped at 2^24).
    r = rng(31)
    a = np.arange(1 << 24, dtype=np.float64) * 2.0 ** -24
    u = a.astype(np.float32)
    for _ in range(4):
        p_x = np.float32(r.random() * 0.5)
        q_x = np.float32(r.random() * 0.5 + 0.1)
        count = int(np.sum(oracle.accept_flags(np.full_like(u, p_x), np.full_like(u, q_x), u)))
        expect = min(1 << 24, math.ceil(Fraction(float(p_x)) / Fraction(float(q_x)) * (1 << 24)))
        assert count == expect


def test_accept_greedy_planted_mismatch():
    r = rng(32)
    k, V = 5, 40
    for m in range(k + 1):
        p = _random_probs(r, (k + 1, V))
        g = np.argmax(p, axis=-1)
        draft = [int(x) for x in g[:k]]
        if m < k:
            draft[m] = (draft[m] + 1) % V
        n, toks = oracle.spec_accept_one(p, None, draft, None, oracle.ACCEPT_GREEDY)
        assert n == m
        assert toks[:m] == draft[:m] and toks[m] == int(g[m])
        assert toks[m + 1:] == [-1] * (k - m)


def test_accept_invalid_draft_id_is_rejected():
    p = np.full((3, 4), 0.25, dtype=np.float32)
    n, toks = oracle.spec_accept_one(p, p[:2], [7, 1], np.zeros(3, np.float32), oracle.ACCEPT_SAMPLED)
    assert n == 0 and 0 <= toks[0] < 4
    n, toks = oracle.spec_accept_one(p, None, [-1, 1], None, oracle.ACCEPT_GREEDY)
    assert n == 0 and toks[0] == 0


def test_residual_weights_fixed_point():
    # exactly representable differences map to exact integers; anything
    # below 2^-40 weighs zero; negatives clamp to zero
    p = np.array([0.75, 0.25, 2.0 ** -41, 0.0, 2.0 ** -40], dtype=np.float32)
    q = np.array([0.25, 0.5, 0.0, 0.0, 0.0], dtype=np.float32)
    R = oracle.residual_weights(p, q)
    assert list(R) == [2 ** 39, 0, 0, 0, 1]
    # fp32 rounding of the subtraction: 1 - 2^-30 rounds to 1 in float32
    R2 = oracle.residual_weights(np.array([1.0], np.float32), np.array([2.0 ** -30], np.float32))
    assert list(R2) == [2 ** 40]


def test_residual_weights_clamp_above_one():
    # Probabilities lie in [0, 1]; a value above 1 (invalid input, used as
    # given rather than renormalised) weighs exactly as 1, i.e. 2^40.  Hand
    # values: residuals [3 - 1, 1.5 - 0, 0.5 - 0] = [2, 1.5, 0.5] give
    # [2^40, 2^40, 2^39]; the bonus weights of [1.25, 0.5, 4.0] (no q) give
    # [2^40, 2^39, 2^40].
    p = np.array([3.0, 1.5, 0.5], np.float32)
    q = np.array([1.0, 0.0, 0.0], np.float32)
    assert list(oracle.residual_weights(p, q)) == [2 ** 40, 2 ** 40, 2 ** 39]
    assert list(oracle.residual_weights(np.array([1.25, 0.5, 4.0], np.float32))) == \
        [2 ** 40, 2 ** 39, 2 ** 40]
    # A row [3, 1] then draws either token with probability exactly 1/2:
    # S = 2^41, T = a * 2^17, token 0 iff T < 2^40 iff a < 2^23.
    R = oracle.residual_weights(np.array([3.0, 1.0], np.float32))
    assert oracle.fixed_point_sample(R, (1 << 23) - 1) == 0
    assert oracle.fixed_point_sample(R, 1 << 23) == 1
    # Through the whole rule: the draft (token 0, q = 1) is rejected by
    # u = 0.75 only if 0.75 * 1 >= p = 3 -- it is accepted, so the final
    # draw comes from the bonus row p_1 = [5, 0.25]: weights [2^40, 2^38],
    # S = 1.25 * 2^40, u_1 = 0.5 gives T = 0.625 * 2^40 < 2^40: token 0.
    pr = np.array([[[3.0, 0.0], [5.0, 0.25]]], np.float32)
    qr = np.array([[[1.0, 0.0]]], np.float32)
    n, tok = oracle.spec_accept(pr, qr, np.array([[0]], np.int32),
                                np.array([[0.75, 0.5]], np.float32), oracle.ACCEPT_SAMPLED)
    assert int(n[0]) == 1 and list(tok[0]) == [0, 0]
    # u_1 = 0.9: T = floor(0.9 * 2^24) * 1.25 * 2^40 / 2^24 >= 2^40: token 1
    n, tok = oracle.spec_accept(pr, qr, np.array([[0]], np.int32),
                                np.array([[0.75, 0.9]], np.float32), oracle.ACCEPT_SAMPLED)
    assert int(n[0]) == 1 and list(tok[0]) == [0, 1]


def test_fixed_point_sample_matches_python_integers():
    r = rng(33)
    R = r.integers(0, 2 ** 40, size=300).astype(np.uint64)
    R[r.integers(0, 300, size=100)] = 0
    S = int(sum(int(x) for x in R))
    cum = np.cumsum([int(x) for x in R])
    for a in list(r.integers(0, 1 << 24, size=200)) + [0, (1 << 24) - 1]:
        T = (int(a) * S) >> 24
        expect = next(j for j in range(len(R)) if int(cum[j]) > T)
        assert oracle.fixed_point_sample(R, int(a)) == expect


def test_fixed_point_sample_exhaustive_counts():
    # All 2^24 uniforms: each token is drawn exactly
    # ceil(c_t 2^24 / S) - ceil(c_{t-1} 2^24 / S) times (c = prefix sums),
    # and a token of zero weight is never drawn.
    r = rng(34)
    V = 16
    R = r.integers(0, 2 ** 40, size=V).astype(np.uint64)
    R[[3, 7, 8]] = 0
    S = int(sum(int(x) for x in R))
    toks = oracle.fixed_point_sample(R, np.arange(1 << 24, dtype=np.uint64))
    counts = np.bincount(toks, minlength=V)
    prev = 0
    c = 0
    for t in range(V):
        c += int(R[t])
        hi = -((-c * (1 << 24)) // S)
        assert counts[t] == hi - prev, t
        prev = hi
    assert counts[[3, 7, 8]].sum() == 0


def _exact_first_token_distribution(p, q):
    """Exact distribution of the first output token, k = 1, draft x ~ q.

    Enumerates every uniform on the 2^-24 grid through the oracle's own
    acceptance test and final draw.
    """
    V = p.shape[1]
    grid = (np.arange(1 << 24, dtype=np.float64) * 2.0 ** -24).astype(np.float32)
    R = oracle.residual_weights(p[0], q[0])
    rho = np.bincount(oracle.fixed_point_sample(R, np.arange(1 << 24, dtype=np.uint64)),
                      minlength=V)
    dist = [Fraction(0)] * V
    for x in range(V):
        acc = int(np.sum(oracle.accept_flags(np.full_like(grid, p[0, x]),
                                             np.full_like(grid, q[0, x]), grid)))
        alpha = Fraction(acc, 1 << 24)
        qx = Fraction(float(q[0, x]))
        dist[x] += qx * alpha
        for t in range(V):
            dist[t] += qx * (1 - alpha) * Fraction(int(rho[t]), 1 << 24)
    return dist


def test_accept_output_distribution_is_the_target_exactly():
    # Speculative sampling leaves the target distribution unchanged
    # (Sec. 3.1 and the rule it cites).  With dyadic p, q summing to 1, the
    # implementation's exact output law differs from p only by the 2^-24
    # grids of the acceptance test and of the final draw: at most 3 * 2^-24.
    r = rng(35)
    V = 16
    for trial in range(2):
        P = r.multinomial(1 << 20, r.dirichlet(np.ones(V) * 0.7))
        Q = r.multinomial(1 << 20, r.dirichlet(np.ones(V) * 0.7))
        p = np.stack([P, P]).astype(np.float64) / (1 << 20)
        q = (Q.astype(np.float64) / (1 << 20))[None]
        p = p.astype(np.float32)
        q = q.astype(np.float32)
        # the ideal rule with exact rationals reproduces p exactly
        pf = [Fraction(int(x), 1 << 20) for x in P]
        qf = [Fraction(int(x), 1 << 20) for x in Q]
        beta = sum(min(a, b) for a, b in zip(pf, qf))
        resid = [max(Fraction(0), a - b) for a, b in zip(pf, qf)]
        zr = sum(resid)
        ideal = [qf[t] * min(Fraction(1), pf[t] / qf[t]) if qf[t] > 0 else Fraction(0)
                 for t in range(V)]
        ideal = [ideal[t] + (1 - beta) * resid[t] / zr for t in range(V)]
        assert ideal == pf
        dist = _exact_first_token_distribution(p, q)
        assert sum(dist) == 1
        worst = max(abs(dist[t] - pf[t]) for t in range(V))
        assert worst <= Fraction(3, 1 << 24), float(worst)


def test_accept_monte_carlo_first_token_law():
    # The composed per-sequence rule (tests, rejection, final draw with the
    # last uniform) reproduces p for the first output token.
    r = rng(36)
    V, k, n_samp = 12, 2, 12000
    p = _random_probs(r, (k + 1, V))
    q = _random_probs(r, (k, V))
    counts = np.zeros(V)
    for _ in range(n_samp):
        c = np.cumsum(q[0].astype(np.float64))
        x0 = min(V - 1, int(np.searchsorted(c, r.random() * c[-1], side="right")))
        c1 = np.cumsum(q[1].astype(np.float64))
        x1 = min(V - 1, int(np.searchsorted(c1, r.random() * c1[-1], side="right")))
        u = (r.integers(0, 1 << 24, size=k + 1) * 2.0 ** -24).astype(np.float32)
        _, toks = oracle.spec_accept_one(p, q, [x0, x1], u, oracle.ACCEPT_SAMPLED)
        counts[toks[0]] += 1
    expect = p[0].astype(np.float64) * n_samp
    chi2 = float(np.sum((counts - expect) ** 2 / np.maximum(expect, 1e-9)))
    # chi-square with 11 degrees of freedom: P(chi2 > 31.3) ~ 0.001
    assert chi2 < 31.3, chi2


def test_accept_uniform_roles():
    # u_0..u_{k-1} drive the tests and u_k the final draw: moving u_0 inside
    # the accepting range leaves the output alone; u_k never changes n.
    p = np.array([[0.5, 0.5, 0, 0], [0.1, 0.2, 0.3, 0.4]], dtype=np.float32)
    q = np.array([[0.25, 0.75, 0, 0]], dtype=np.float32)
    outs = set()
    for u0 in [0.0, 0.3, 0.6]:
        outs.add(tuple(oracle.spec_accept_one(p, q, [1], np.array([u0, 0.55], np.float32),
                                              oracle.ACCEPT_SAMPLED)[1]))
    assert len(outs) == 1
    ns = {oracle.spec_accept_one(p, q, [1], np.array([0.9, uk], np.float32),
                                 oracle.ACCEPT_SAMPLED)[0] for uk in [0.0, 0.4, 0.99]}
    assert ns == {0}


def test_accept_degenerate_residual_falls_back():
    # Unnormalised rows: p <= q everywhere on a rejected row leaves no
    # residual mass; the draw then uses p_n itself, then argmax.
    p = np.array([[0.1, 0.2, 0.1], [0.3, 0.3, 0.4]], dtype=np.float32)
    q = np.array([[0.5, 0.5, 0.5]], dtype=np.float32)
    n, toks = oracle.spec_accept_one(p, q, [1], np.array([0.99, 0.0], np.float32),
                                     oracle.ACCEPT_SAMPLED)
    assert n == 0 and toks[0] == 0           # a = 0 picks the first weighted token
    n, toks = oracle.spec_accept_one(p, q, [1], np.array([0.99, 0.99], np.float32),
                                     oracle.ACCEPT_SAMPLED)
    assert n == 0 and toks[0] == 2
    z = np.zeros((2, 3), dtype=np.float32)
    n, toks = oracle.spec_accept_one(z, q, [1], np.array([0.5, 0.5], np.float32),
                                     oracle.ACCEPT_SAMPLED)
    assert n == 0 and toks[0] == 0


def test_accept_batch_matches_per_sequence():
    r = rng(37)
    B, k, V = 3, 4, 30
    p = _random_probs(r, (B, k + 1, V))
    q = _random_probs(r, (B, k, V))
    d = r.integers(0, V, size=(B, k)).astype(np.int32)
    u = (r.integers(0, 1 << 24, size=(B, k + 1)) * 2.0 ** -24).astype(np.float32)
    n, t = oracle.spec_accept(p, q, d, u, oracle.ACCEPT_SAMPLED)
    for b in range(B):
        nb, tb = oracle.spec_accept_one(p[b], q[b], d[b], u[b], oracle.ACCEPT_SAMPLED)
        assert n[b] == nb and list(t[b]) == tb


# ---------------------------------------------------------------- LM head
# Sec. 3.1 (the head maps a feature to a vocabulary distribution), Sec. 3.3
# and Algorithm 1 (the draft's states projected by the same head, drafts
# drawn from the result), Sec. 4.2 (temperature).

def test_lm_head_zero_weights_give_uniform():
    r = rng(41)
    h = r.standard_normal((3, 8))
    p = oracle.lm_head_probs(h, np.zeros((7, 8)), 0.7)
    assert np.allclose(p, 1.0 / 7, atol=1e-15)


def test_lm_head_two_token_logistic_closed_form():
    # V = 2: p_1 = 1 / (1 + exp((z_0 - z_1) / tau)); pins the orientation
    # (logit v = h . W[v]) and that the logits are divided by tau.
    h = np.array([[1.5, -2.0, 0.25]])
    w = np.array([[0.5, 1.0, 2.0], [-1.0, 0.5, 4.0]])
    z0 = 1.5 * 0.5 - 2.0 * 1.0 + 0.25 * 2.0
    z1 = 1.5 * -1.0 - 2.0 * 0.5 + 0.25 * 4.0
    for tau in (0.5, 1.0, 3.0):
        p = oracle.lm_head_probs(h, w, tau)[0]
        want = 1.0 / (1.0 + math.exp((z0 - z1) / tau))
        assert abs(p[1] - want) < 1e-15 and abs(p[0] - (1.0 - want)) < 1e-15


def test_lm_head_temperature_is_a_power_law():
    # softmax(z / tau) is proportional to softmax(z)^(1 / tau)
    r = rng(42)
    h, w = r.standard_normal((2, 6)), r.standard_normal((9, 6))
    p1 = oracle.lm_head_probs(h, w, 1.0)
    for tau in (0.35, 0.7, 2.5):
        pt = oracle.lm_head_probs(h, w, tau)
        q = p1 ** (1.0 / tau)
        assert np.allclose(pt, q / q.sum(axis=1, keepdims=True), rtol=1e-12, atol=1e-300)


def test_lm_head_temperature_limits():
    h = np.array([[1.0, 0.0]])
    w = np.array([[0.3, 0.0], [0.9, 0.0], [0.1, 0.0]])
    assert np.allclose(oracle.lm_head_probs(h, w, 1e7), 1.0 / 3, atol=1e-7)
    p = oracle.lm_head_probs(h, w, 1e-3)
    assert p[0, 1] > 1 - 1e-12 and np.argmax(p[0]) == 1


def test_lm_head_shift_and_permutation():
    r = rng(43)
    h, w = r.standard_normal((3, 5)), r.standard_normal((11, 5))
    p = oracle.lm_head_probs(h, w, 0.8)
    # a constant added to every logit (an extra feature of 1 against a
    # weight column of 2.5) changes nothing
    h2 = np.concatenate([h, np.ones((3, 1))], axis=1)
    w2 = np.concatenate([w, np.full((11, 1), 2.5)], axis=1)
    assert np.allclose(oracle.lm_head_probs(h2, w2, 0.8), p, rtol=1e-12)
    perm = r.permutation(11)
    assert np.allclose(oracle.lm_head_probs(h, w[perm], 0.8), p[:, perm], rtol=1e-14)
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-14)


def test_lm_head_brute_force_tiny():
    r = rng(44)
    R, d, V, tau = 2, 3, 4, 0.6
    h, w = r.standard_normal((R, d)), r.standard_normal((V, d))
    got = oracle.lm_head_probs(h, w, tau)
    for i in range(R):
        z = [sum(h[i][j] * w[v][j] for j in range(d)) / tau for v in range(V)]
        m = max(z)
        e = [math.exp(x - m) for x in z]
        for v in range(V):
            assert abs(got[i][v] - e[v] / sum(e)) < 1e-14


def test_sample_tokens_dyadic_thresholds():
    # p = (1/4, 1/2, 1/8, 1/8): weights are exact, S = 2^40, T = a * 2^16,
    # so the token changes exactly at u = 1/4, 3/4 and 7/8
    p = np.array([[0.25, 0.5, 0.125, 0.125]] * 7, dtype=np.float32)
    u = np.array([0.0, 0.25 - 2 ** -24, 0.25, 0.75 - 2 ** -24, 0.75, 0.875, 1 - 2 ** -24],
                 dtype=np.float32)
    assert list(oracle.sample_tokens(p, u)) == [0, 0, 1, 1, 2, 3, 3]


def test_sample_tokens_one_hot_and_degenerate():
    p = np.zeros((3, 5), dtype=np.float32)
    p[0, 3] = 1.0
    p[1, 1] = 1e-13                     # below 2^-40: no weight, argmax decides
    p[1, 4] = 5e-13
    u = np.array([0.9, 0.1, 0.3], dtype=np.float32)
    assert list(oracle.sample_tokens(p, u)) == [3, 4, 0]


# ------------------------------------------------- acceptance from logits

def _numpy_philox_block(counter, key):
    """The block numpy's independent Philox-4x64 implementation produces at
    256-bit counter `counter` (numpy advances its counter before each block,
    so it is started one below)."""
    c = sum(int(x) << (64 * i) for i, x in enumerate(counter)) - 1
    c %= 1 << 256
    start = np.array([(c >> (64 * i)) & ((1 << 64) - 1) for i in range(4)], dtype=np.uint64)
    g = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=start)
    return [int(x) for x in g.random_raw(4)]


def test_philox_matches_numpy_implementation():
    cases = [((0, 0, 0, 0), (0, 0)), ((1, 2, 3, 4), (5, 6)), ((0, 7, 1, 0), (123456789, 0)),
             ((2 ** 64 - 1, 3, 0, 0), (2 ** 63 + 11, 99)), ((5, 0, 2 ** 40, 0), (2 ** 64 - 1, 2 ** 64 - 1))]
    for ctr, key in cases:
        assert oracle.philox4x64(ctr, key) == _numpy_philox_block(ctr, key), (ctr, key)


def test_philox_uniforms_layout_and_grid():
    seed, offset, B, n = 0x1234ABCD, 77, 3, 9
    u = oracle.philox_uniforms(seed, offset, B, n)
    assert u.shape == (B, n) and u.dtype == np.float32
    a = u.astype(np.float64) * 2.0 ** 24
    assert np.all(a == np.floor(a)) and np.all((a >= 0) & (a < 2 ** 24))
    for b in range(B):
        for i in range(n):
            word = _numpy_philox_block((i // 4, b, offset, 0), (seed, 0))[i % 4]
            assert int(a[b, i]) == word >> 40
    # different seeds, offsets and sequences give different streams
    assert not np.array_equal(u, oracle.philox_uniforms(seed + 1, offset, B, n))
    assert not np.array_equal(u, oracle.philox_uniforms(seed, offset + 1, B, n))
    assert not np.array_equal(u[0], u[1])


def _logit_case(seed, B=2, k=3, V=11, scale=3.0, integer=False):
    rng = np.random.default_rng(seed)
    z = rng.normal(size=(B, k + 1, V)) * scale
    zd = z[:, :k] + rng.normal(size=(B, k, V))
    if integer:
        z, zd = np.round(z), np.round(zd)
    draft = rng.integers(0, V, size=(B, k)).astype(np.int32)
    return z, zd, draft


def test_accept_logits_scale_and_shift_invariance():
    # softmax(z / tau) is unchanged (exactly, in binary floating point) by a
    # power-of-two scale of both z and tau, and by integer shifts of a row of
    # integer-valued logits
    z, zd, draft = _logit_case(5, integer=True)
    ref = oracle.spec_accept_logits(z, zd, draft, 9, 1, 0.75, oracle.ACCEPT_SAMPLED)
    scaled = oracle.spec_accept_logits(4 * z, 4 * zd, draft, 9, 1, 3.0, oracle.ACCEPT_SAMPLED)
    shift = np.arange(z.shape[1])[None, :, None] * 7.0
    shifted = oracle.spec_accept_logits(z + shift, zd - shift[:, :-1], draft, 9, 1, 0.75,
                                        oracle.ACCEPT_SAMPLED)
    for got in (scaled, shifted):
        assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])


def test_accept_logits_cold_limit_is_greedy():
    # as tau -> 0, p and q become one-hot at the argmaxes: a draft equal to
    # the target argmax is accepted (u q = u < 1 = p), any other is rejected
    # (p = 0) and the residual is one-hot at the target argmax
    z, zd, _ = _logit_case(11, B=4, k=4, V=13)
    draft = np.argmax(zd, axis=-1).astype(np.int32)
    draft[1, 0] = np.argmax(z[1, 0])                     # plant agreements
    draft[2, :2] = np.argmax(z[2, :2], axis=-1)
    cold = oracle.spec_accept_logits(z, zd, draft, 3, 0, 1e-4, oracle.ACCEPT_SAMPLED)
    greedy = oracle.spec_accept_logits(z, None, draft, 0, 0, 0.0, oracle.ACCEPT_GREEDY)
    assert np.array_equal(cold[0], greedy[0]) and np.array_equal(cold[1], greedy[1])


def test_accept_logits_greedy_ignores_temperature_and_seed():
    z, zd, _ = _logit_case(2, B=3, k=3, V=9)
    draft = np.argmax(z[:, :3], axis=-1).astype(np.int32)
    draft[0, 1] = (draft[0, 1] + 1) % 9                  # mismatch at position 1
    a = oracle.spec_accept_logits(z, zd, draft, 1, 2, 0.3, oracle.ACCEPT_GREEDY)
    b = oracle.spec_accept_logits(z, None, draft, 8, 5, 2.0, oracle.ACCEPT_GREEDY)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert a[0].tolist() == [1, 3, 3]
    assert a[1][0].tolist()[:2] == [draft[0, 0], int(np.argmax(z[0, 1]))]


def test_accept_logits_first_token_follows_target_law():
    # speculative sampling emits its first token with the target law p_0
    # whatever the draft does; over many (seed, offset) streams the counts
    # pass a chi-square test against softmax(z_0 / tau)
    V, k, tau = 6, 2, 1.3
    rng = np.random.default_rng(4)
    z = rng.normal(size=(1, k + 1, V)) * 1.5
    zd = rng.normal(size=(1, k, V)) * 1.5
    q = oracle.softmax_temperature(zd, tau)
    p0 = oracle.softmax_temperature(z, tau)[0, 0]
    counts = np.zeros(V)
    trials = 6000
    for s in range(trials):
        # the drafts follow q (drawn from an unrelated generator)
        d = np.array([[rng.choice(V, p=q[0, i]) for i in range(k)]], dtype=np.int32)
        n, toks = oracle.spec_accept_logits(z, zd, d, 1000 + s, s, tau, oracle.ACCEPT_SAMPLED)
        counts[toks[0, 0]] += 1
    expected = p0 * trials
    chi2 = float(np.sum((counts - expected) ** 2 / expected))
    # 5 degrees of freedom: P(chi2 > 20.5) ~ 0.001
    assert chi2 < 20.5, (counts, expected)


# ---------------------------------------------------------------- draft layer
def test_rms_norm_closed_forms():
    w = np.array([0.5, -2.0, 3.0, 1.0])
    # a constant row c * 1 has rms |c|: the output is sign(c) * w (eps = 0)
    assert np.allclose(oracle.rms_norm(np.full(4, -7.0), w, 0.0), -w, rtol=0, atol=1e-15)
    # [3, 4] has mean square 12.5
    r = math.sqrt(12.5)
    assert np.allclose(oracle.rms_norm(np.array([3.0, 4.0]), np.ones(2), 0.0), [3 / r, 4 / r], atol=1e-15)
    # eps enters under the root: [1, 1] with eps = 3 is divided by 2
    assert np.allclose(oracle.rms_norm(np.array([1.0, 1.0]), np.ones(2), 3.0), [0.5, 0.5], atol=1e-15)
    # invariant under positive scaling (eps = 0), rows independent
    x = np.random.default_rng(0).normal(size=(3, 8))
    assert np.allclose(oracle.rms_norm(x * 9.5, np.ones(8), 0.0), oracle.rms_norm(x, np.ones(8), 0.0))


def test_rope_closed_forms_and_relative_position():
    # D = 2: (1, 0) at position p becomes (cos p, sin p)
    for p in [0, 1, 5, 37]:
        assert np.allclose(oracle.rope(np.array([[1.0, 0.0]]), np.array([p]), 10000.0),
                           [[math.cos(p), math.sin(p)]], atol=1e-14)
    # D = 4, theta = 10000: pair 1 turns at 10000^(-1/2) = 0.01 rad per position
    y = oracle.rope(np.array([[0.0, 1.0, 0.0, 0.0]]), np.array([50]), 10000.0)
    assert np.allclose(y, [[0.0, math.cos(0.5), 0.0, math.sin(0.5)]], atol=1e-14)
    rng = np.random.default_rng(1)
    x = rng.normal(size=(6, 8))
    # position 0 is the identity; every pair keeps its length
    assert np.allclose(oracle.rope(x, np.zeros(6), 500.0), x, atol=0)
    y = oracle.rope(x, np.arange(6) * 3, 500.0)
    assert np.allclose(y[:, :4] ** 2 + y[:, 4:] ** 2, x[:, :4] ** 2 + x[:, 4:] ** 2)
    # scores depend on positions only through their difference
    q, k = rng.normal(size=8), rng.normal(size=8)
    s = lambda m, n: float(oracle.rope(q[None], np.array([m]), 500.0)[0] @ oracle.rope(k[None], np.array([n]), 500.0)[0])
    assert abs(s(9, 4) - s(15, 10)) < 1e-12 and abs(s(3, 3) - float(q @ k)) < 1e-12
    # a heads axis: [n, H, D] with one position per row rotates every head alike
    xh = rng.normal(size=(4, 3, 8))
    yh = oracle.rope(xh, np.arange(4), 500.0)
    for h in range(3):
        assert np.allclose(yh[:, h], oracle.rope(xh[:, h], np.arange(4), 500.0))


def test_linear_and_swiglu_closed_forms():
    rng = np.random.default_rng(2)
    x = rng.normal(size=(3, 5))
    assert np.array_equal(oracle.linear(x, np.eye(5)), x)
    assert np.allclose(oracle.linear(x, np.eye(5)[[4, 0]], bias=[1.0, 2.0], residual=np.ones((3, 2))),
                       np.stack([x[:, 4] + 2.0, x[:, 0] + 3.0], axis=1))
    # silu(0) = 0; silu(x) - silu(-x) = x; sigmoid(log 3) = 3/4
    assert oracle.silu(0.0) == 0.0
    z = rng.normal(size=7) * 4
    assert np.allclose(oracle.silu(z) - oracle.silu(-z), z)
    assert abs(float(oracle.swiglu(np.array([math.log(3.0), 2.0]))[0]) - 0.75 * math.log(3.0) * 2.0) < 1e-15


def _draft_case(seed, B=2, r=3, d=8, hq=2, hkv=1, I=6, ctx=(4, 2), Lmax=10):
    rng = np.random.default_rng(seed)
    D = d // hq
    W = {"fc_w": rng.normal(size=(d, 2 * d)) / 4, "fc_b": rng.normal(size=d),
         "ln1": 1 + rng.normal(size=d) / 5, "wqkv": rng.normal(size=((hq + 2 * hkv) * D, d)) / 3,
         "wo": rng.normal(size=(d, hq * D)) / 3, "ln2": 1 + rng.normal(size=d) / 5,
         "wgu": rng.normal(size=(2 * I, d)) / 3, "wdown": rng.normal(size=(d, I)) / 3}
    u = rng.normal(size=(B, r, 2 * d))
    kc = rng.normal(size=(B, Lmax, hkv, D))
    vc = rng.normal(size=(B, Lmax, hkv, D))
    return u, W, kc, vc, np.array(ctx[:B])


def test_draft_layer_without_branches_is_the_fc_map():
    # Wo = Wdown = 0: the output is FC(u) and the caches gain RoPE(k), v of
    # the normed rows at positions pos .. pos + r - 1, nothing else changes
    u, W, kc, vc, pos = _draft_case(3)
    W0 = dict(W, wo=np.zeros_like(W["wo"]), wdown=np.zeros_like(W["wdown"]))
    out, kc2, vc2 = oracle.semi_ar_layer(u, W0, kc, vc, pos, 2, 1, 1e-6, 10000.0)
    x0 = u @ W["fc_w"].T + W["fc_b"]
    assert np.allclose(out, x0)
    h = x0 / np.sqrt(np.mean(x0 ** 2, axis=-1, keepdims=True) + 1e-6) * W["ln1"]
    kv = h @ W["wqkv"].T                                   # [B, r, 4 * D], D = 4
    for b in range(2):
        p = pos[b]
        assert np.allclose(vc2[b, p:p + 3, 0], kv[b, :, 12:16])
        assert np.allclose(kc2[b, p:p + 3, 0], oracle.rope(kv[b, :, 8:12], p + np.arange(3), 10000.0))
        assert np.array_equal(kc2[b, :p], kc[b, :p]) and np.array_equal(vc2[b, p + 3:], vc[b, p + 3:])


def test_draft_layer_is_causal_inside_the_new_rows():
    # changing row j's input leaves rows < j and other sequences unchanged
    u, W, kc, vc, pos = _draft_case(4)
    ref, _, _ = oracle.semi_ar_layer(u, W, kc, vc, pos, 2, 1, 1e-6, 10000.0)
    u2 = u.copy()
    u2[0, 1] += 1.0
    out, _, _ = oracle.semi_ar_layer(u2, W, kc, vc, pos, 2, 1, 1e-6, 10000.0)
    assert np.allclose(out[0, 0], ref[0, 0]) and np.allclose(out[1], ref[1])
    assert not np.allclose(out[0, 1], ref[0, 1]) and not np.allclose(out[0, 2], ref[0, 2])
    # context entries at or past pos + r are never read
    kc3, vc3 = kc.copy(), vc.copy()
    kc3[0, pos[0] + 3:] = 1e6
    vc3[0, pos[0] + 3:] = -1e6
    out3, _, _ = oracle.semi_ar_layer(u, W, kc3, vc3, pos, 2, 1, 1e-6, 10000.0)
    assert np.allclose(out3, ref)


def test_draft_layer_gqa_equals_repeated_heads():
    # Hkv = 1 shared by 2 query heads equals Hkv = 2 with the KV head repeated
    u, W, kc, vc, pos = _draft_case(5)
    ref, _, _ = oracle.semi_ar_layer(u, W, kc, vc, pos, 2, 1, 1e-6, 10000.0)
    D = 4
    wq, wk, wv = W["wqkv"][:2 * D], W["wqkv"][2 * D:3 * D], W["wqkv"][3 * D:]
    W2 = dict(W, wqkv=np.concatenate([wq, wk, wk, wv, wv]))
    out, _, _ = oracle.semi_ar_layer(u, W2, np.repeat(kc, 2, axis=2), np.repeat(vc, 2, axis=2), pos, 2, 2,
                                     1e-6, 10000.0)
    assert np.allclose(out, ref)


def test_draft_layer_brute_force():
    # pure-Python loops on a tiny case: d = 4, 2 heads of D = 2, I = 3
    u, W, kc, vc, pos = _draft_case(6, B=1, r=2, d=4, hq=2, hkv=2, I=3, ctx=(3,), Lmax=6)
    out, _, _ = oracle.semi_ar_layer(u, W, kc, vc, pos, 2, 2, 1e-5, 100.0)
    d, D, I, eps, theta = 4, 2, 3, 1e-5, 100.0
    L = W["wqkv"].tolist()

    def mv(m, x):
        return [sum(m[i][j] * x[j] for j in range(len(x))) for i in range(len(m))]

    def norm(x, w):
        r = math.sqrt(sum(v * v for v in x) / len(x) + eps)
        return [x[i] / r * w[i] for i in range(len(x))]

    def rot(x, p):                             # D = 2: one pair, frequency 1
        return [x[0] * math.cos(p) - x[1] * math.sin(p), x[1] * math.cos(p) + x[0] * math.sin(p)]

    keys = {t: [list(kc[0, t, h]) for h in range(2)] for t in range(pos[0])}
    vals = {t: [list(vc[0, t, h]) for h in range(2)] for t in range(pos[0])}
    xs = []
    for j in range(2):
        x0 = [v + b for v, b in zip(mv(W["fc_w"].tolist(), u[0, j].tolist()), W["fc_b"].tolist())]
        qkv = mv(L, norm(x0, W["ln1"].tolist()))
        p = pos[0] + j
        keys[p] = [rot(qkv[4 + 2 * h:6 + 2 * h], p) for h in range(2)]
        vals[p] = [qkv[8 + 2 * h:10 + 2 * h] for h in range(2)]
        xs.append((x0, [rot(qkv[2 * h:2 * h + 2], p) for h in range(2)], p))
    for j, (x0, qs, p) in enumerate(xs):
        att = []
        for h in range(2):
            s = [(qs[h][0] * keys[t][h][0] + qs[h][1] * keys[t][h][1]) / math.sqrt(D) for t in range(p + 1)]
            m = max(s)
            e = [math.exp(v - m) for v in s]
            att += [sum(e[t] * vals[t][h][c] for t in range(p + 1)) / sum(e) for c in range(2)]
        x1 = [a + b for a, b in zip(x0, mv(W["wo"].tolist(), att))]
        gu = mv(W["wgu"].tolist(), norm(x1, W["ln2"].tolist()))
        act = [gu[i] / (1 + math.exp(-gu[i])) * gu[I + i] for i in range(I)]
        x2 = [a + b for a, b in zip(x1, mv(W["wdown"].tolist(), act))]
        assert np.allclose(out[0, j], x2, rtol=1e-12, atol=1e-12), j


def _kp_case(seed, B=2, r0=3, kp=2, d=8, V=11):
    u0, W, kc, vc, pos = _draft_case(seed, B=B, r=r0, Lmax=16)
    rng = np.random.default_rng(seed + 100)
    u0 = u0.copy()
    ph = rng.normal(size=2 * d)
    u0[:, r0 - kp:] = ph                                   # the last k' rows are placeholders
    lm_w = rng.normal(size=(V, d)) * 3 / np.sqrt(d)
    emb = rng.normal(size=(V, d))
    return u0, W, kc, vc, pos, ph, lm_w, emb


def test_bf16_round_matches_hand_values():
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: ties go to the even mantissa (1)
    assert oracle.bf16_round(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    assert oracle.bf16_round(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6
    assert oracle.bf16_round(np.array([-2.5]))[0] == -2.5            # exact
    assert oracle.bf16_round(np.array([1.0 + 2.0 ** -9]))[0] == 1.0  # below half an ulp


def test_kp_draft_single_pass_is_layer_head_and_draw():
    # k' = K: one pass; the drafts are the head's draws from the placeholder rows
    u0, W, kc, vc, pos, ph, lm_w, emb = _kp_case(7, r0=3, kp=2)
    uni = (np.arange(4).reshape(2, 2) * 2 ** 21 * 2.0 ** -24 + 0.1).astype(np.float32)
    tok, q = oracle.semi_ar_draft(u0, W, lm_w, emb, ph, kc, vc, pos, 2, 1, 1e-6, 1e4, 0.8, uni, 2, 2)
    out, _, _ = oracle.semi_ar_layer(u0, W, kc, vc, pos, 2, 1, 1e-6, 1e4)
    p = oracle.lm_head_probs(oracle.bf16_round(out[:, 1:]).reshape(4, 8), lm_w, 0.8)
    assert np.allclose(q.reshape(4, -1), p)
    assert np.array_equal(tok.reshape(-1), oracle.sample_tokens(p.astype(np.float32), uni.reshape(-1)))


def test_kp_draft_first_draft_independent_of_group_size():
    # the first placeholder sees only the rows before it (causal), so its
    # distribution is the same for every k'
    u0, W, kc, vc, pos, ph, lm_w, emb = _kp_case(8, r0=5, kp=4)
    uni = np.full((2, 4), 0.37, dtype=np.float32)
    qs = []
    for kp in (1, 2, 4):
        u = u0[:, :1 + kp].copy()                          # one text row + k' placeholders
        _, q = oracle.semi_ar_draft(u, W, lm_w, emb, ph, kc, vc, pos, 2, 1, 1e-6, 1e4, 1.0, uni, 4, kp)
        qs.append(q)
    assert np.allclose(qs[0][:, 0], qs[1][:, 0]) and np.allclose(qs[0][:, 0], qs[2][:, 0])
    assert not np.allclose(qs[0][:, 1], qs[2][:, 1])       # later drafts do depend on k'


def test_kp_draft_feeds_drafts_back_in_order():
    # forced tokens: the distributions of pass t depend on the tokens of
    # passes < t only; a later pass's uniforms never change earlier drafts
    u0, W, kc, vc, pos, ph, lm_w, emb = _kp_case(9, r0=3, kp=2)
    uni = np.full((2, 6), 0.5, dtype=np.float32)
    forced = np.array([[1, 2, 3, 4, 5, 6], [7, 8, 9, 10, 0, 1]], dtype=np.int32)
    _, qa = oracle.semi_ar_draft(u0, W, lm_w, emb, ph, kc, vc, pos, 2, 1, 1e-6, 1e4, 1.0, uni, 6, 2, forced)
    f2 = forced.copy()
    f2[:, 2] = (f2[:, 2] + 1) % 11                          # change a draft of pass 1
    _, qb = oracle.semi_ar_draft(u0, W, lm_w, emb, ph, kc, vc, pos, 2, 1, 1e-6, 1e4, 1.0, uni, 6, 2, f2)
    assert np.allclose(qa[:, :4], qb[:, :4]) and not np.allclose(qa[:, 4:], qb[:, 4:])
    uni2 = uni.copy()
    uni2[:, 4:] = 0.99
    ta, _ = oracle.semi_ar_draft(u0, W, lm_w, emb, ph, kc, vc, pos, 2, 1, 1e-6, 1e4, 1.0, uni, 6, 2)
    tb, _ = oracle.semi_ar_draft(u0, W, lm_w, emb, ph, kc, vc, pos, 2, 1, 1e-6, 1e4, 1.0, uni2, 6, 2)
    assert np.array_equal(ta[:, :4], tb[:, :4])


def test_int8_rows_dequantise_and_project():
    # W = scale[n] * wq[n, :]: unit scales give the int8 matrix itself; a
    # row of scale 1/2 halves its output column; one-hot int8 rows pick inputs
    wq = np.array([[1, -2, 0], [127, -128, 3]], dtype=np.int8)
    assert np.array_equal(oracle.dequantize_rows(wq, [1.0, 1.0]), wq.astype(np.float64))
    assert np.array_equal(oracle.dequantize_rows(wq, [0.5, 2.0]), [[0.5, -1.0, 0.0], [254.0, -256.0, 6.0]])
    x = np.array([[2.0, 3.0, 5.0]])
    onehot = np.array([[0, 0, 1], [1, 0, 0]], dtype=np.int8)
    assert np.array_equal(oracle.linear_q8(x, onehot, [1.0, 0.25]), [[5.0, 0.5]])
    assert np.array_equal(oracle.linear_q8(x, onehot, [1.0, 1.0], bias=[1.0, -1.0]), [[6.0, 1.0]])


def test_int8_layer_equals_layer_of_dequantised_weights():
    # an int8 draft whose rows are exactly representable equals the float
    # draft with those weights
    u, W, kc, vc, pos = _draft_case(12)
    rng = np.random.default_rng(12)
    Wq = dict(W)
    Wf = dict(W)
    for name in oracle.draft_layer.Q8_WEIGHTS:
        q = rng.integers(-127, 128, size=W[name].shape).astype(np.int8)
        s = rng.uniform(0.001, 0.02, size=W[name].shape[0])
        Wq[name], Wq[name + "_s"] = q, s
        Wf[name] = s[:, None] * q.astype(np.float64)
    a, ka, va = oracle.semi_ar_layer_q8(u, Wq, kc, vc, pos, 2, 1, 1e-6, 1e4)
    b, kb, vb = oracle.semi_ar_layer(u, Wf, kc, vc, pos, 2, 1, 1e-6, 1e4)
    assert np.array_equal(a, b) and np.array_equal(ka, kb) and np.array_equal(va, vb)


def test_compress_q8_dequantisation_hand_values():
    # an int8 row stands for q * 2^e with its own exponent
    q = np.array([[-127, 5, 0], [1, -2, 64]], np.int8)
    e = np.array([-3, 2], np.int8)
    x = oracle.dequantize_pow2_rows(q, e)
    assert x.tolist() == [[-15.875, 0.625, 0.0], [4.0, -8.0, 256.0]]


def test_compress_q8_two_token_closed_form():
    # one latent [1, 0] (q [1, 0], e 0) over tokens [2, 0] (q [1, 0], e 1)
    # and [0, 3] (q [0, 3], e 0), scale 1: scores [2, 0], so
    # out = (e^2 [2, 0] + [0, 3]) / (e^2 + 1)
    out = oracle.latent_compress_q8(np.array([[1, 0]], np.int8), np.array([0], np.int8),
                                    np.array([[[1, 0], [0, 3]]], np.int8), np.array([[1, 0]], np.int8),
                                    1, 1.0)
    e2 = math.exp(2.0)
    expect = np.array([2 * e2, 3.0]) / (e2 + 1.0)
    assert np.allclose(out[0, 0], expect, rtol=1e-15, atol=0)


def test_compress_q8_exponent_shift_doubles_the_output():
    # moving one power of two from every latent row to every token row
    # leaves the scores unchanged and doubles the values: out doubles exactly
    r = rng(71)
    lq = r.integers(-127, 128, size=(6, 16)).astype(np.int8)
    fq = r.integers(-127, 128, size=(2, 9, 16)).astype(np.int8)
    le = r.integers(-7, -3, size=6).astype(np.int8)
    fe = r.integers(-7, -3, size=(2, 9)).astype(np.int8)
    a = oracle.latent_compress_q8(lq, le, fq, fe, 2, 0.5)
    b = oracle.latent_compress_q8(lq, (le - 1).astype(np.int8), fq, (fe + 1).astype(np.int8), 2, 0.5)
    assert np.allclose(b, 2.0 * a, rtol=1e-13, atol=0)


def test_compress_q8_zero_queries_average_the_dequantised_tokens():
    r = rng(72)
    fq = r.integers(-127, 128, size=(1, 5, 8)).astype(np.int8)
    fe = np.array([[-2, 0, 1, -5, 3]], np.int8)
    out = oracle.latent_compress_q8(np.zeros((3, 8), np.int8), np.zeros(3, np.int8), fq, fe, 1, 1.0)
    mean = sum(fq[0, t].astype(np.float64) * 2.0 ** int(fe[0, t]) for t in range(5)) / 5.0
    for c in range(3):
        assert np.allclose(out[0, c], mean, rtol=1e-13, atol=1e-12)


def test_avg_pool_compress_closed_forms():
    rng = np.random.default_rng(21)
    F = rng.normal(size=(2, 7, 5))
    # C = N is the identity, C = 1 the global mean, which is also Eq. 3 with
    # zero queries (every token weighted 1/N)
    assert np.allclose(oracle.avg_pool_compress(F, 7), F)
    g = oracle.avg_pool_compress(F, 1)
    assert np.allclose(g[:, 0], F.mean(axis=1))
    assert np.allclose(np.repeat(g, 3, axis=1), oracle.latent_compress(np.zeros((3, 5)), F, 1, 1.0))
    # N = 7, C = 3: groups floor(7c/3) .. -> tokens {0, 1}, {2, 3}, {4, 5, 6}
    x = np.arange(7, dtype=np.float64).reshape(1, 7, 1)
    assert np.array_equal(oracle.avg_pool_compress(x, 3)[0, :, 0], [0.5, 2.5, 5.0])
