"""Oracle for the verification attention of the drafted block (Sec. 3.1).

Test infrastructure only (see the package docstring).

During verification the target model scores all K drafted tokens in one
forward pass (Sec. 3.1; Sec. 3.3).  Inside each target layer that pass is
ordinary scaled dot-product attention of the K block positions over the KV
cache of the prefix plus the block itself, causal inside the block.  This
module states that attention plainly: it materialises the full score matrix
for every (sequence, query head) and takes a masked softmax.

Readings (the paper names no KV cache, head grouping or mask alignment):
* ``kv_len[b]`` counts every cache entry of sequence b *including* the k
  block entries, which are the last k.  Block row j (0-based) sees keys
  t = 0 .. kv_len[b] - k + j (causal, aligned bottom-right).  A row that
  would see no key (kv_len[b] - k + j < 0) outputs zeros and lse = -inf.
* Grouped-query attention: query head h reads KV head h // (Hq / Hkv).
* Scores are scale * q . k with natural exp / log; callers pass
  scale = 1 / sqrt(D) for standard attention.  q and k are post-RoPE.
* Contiguous cache layout [B, Lmax, Hkv, D]; paged cache layout is a page
  pool [P, Hkv, page_size, D] with page_table[b][t // page_size] naming the
  page that holds token t of sequence b at slot t % page_size.
"""

import numpy as np


def gather_paged(pool, page_table, kv_len, page_size=16):
    """Gather each sequence's logical cache [L_b, Hkv, D] out of a page pool.

    pool: [P, Hkv, page_size, D]; page_table: [B, max_pages] int.
    Returns a list of float64 arrays, one per sequence.
    """
    pool = np.asarray(pool, dtype=np.float64)
    page_table = np.asarray(page_table)
    seqs = []
    for b, L in enumerate(np.asarray(kv_len).tolist()):
        rows = []
        for t in range(L):
            page = int(page_table[b, t // page_size])
            rows.append(pool[page, :, t % page_size, :])
        if rows:
            seqs.append(np.stack(rows, axis=0))
        else:
            seqs.append(np.zeros((0, pool.shape[1], pool.shape[3]), dtype=np.float64))
    return seqs


def verify_attention(q, k_cache, v_cache, kv_len, scale, page_table=None,
                     page_size=16, return_probs=False):
    """Attention of the k-token verification block over the KV cache.

    q:        [B, k, Hq, D] queries of the drafted block (post-RoPE).
    k_cache, v_cache: contiguous [B, Lmax, Hkv, D], or page pools
              [P, Hkv, page_size, D] when ``page_table`` is given.
    kv_len:   [B] cache length of each sequence, block entries included.
    Returns (out [B, k, Hq, D], lse [B, k, Hq]) in float64, where for each
    (b, j, h) with visible keys t <= kv_len[b] - k + j:
        s_t = scale * q[b, j, h] . K[b, t, h // g]
        out = sum_t softmax(s)_t V[b, t, h // g],  lse = log sum_t exp(s_t).
    With ``return_probs`` a list (per b) of [k, Hq, L_b] probabilities is
    appended to the result.
    """
    q = np.asarray(q, dtype=np.float64)
    B, k, Hq, D = q.shape
    kv_len = [int(x) for x in np.asarray(kv_len).reshape(-1).tolist()]
    if len(kv_len) != B:
        raise ValueError("kv_len must hold one length per sequence")
    if page_table is None:
        K = np.asarray(k_cache, dtype=np.float64)
        Vc = np.asarray(v_cache, dtype=np.float64)
        keys = [K[b, :kv_len[b]] for b in range(B)]
        vals = [Vc[b, :kv_len[b]] for b in range(B)]
        Hkv = K.shape[2]
    else:
        keys = gather_paged(k_cache, page_table, kv_len, page_size)
        vals = gather_paged(v_cache, page_table, kv_len, page_size)
        Hkv = np.asarray(k_cache).shape[1]
    if Hq % Hkv != 0:
        raise ValueError("query heads must be a multiple of KV heads")
    g = Hq // Hkv
    out = np.zeros((B, k, Hq, D), dtype=np.float64)
    lse = np.full((B, k, Hq), -np.inf, dtype=np.float64)
    all_probs = []
    for b in range(B):
        L = kv_len[b]
        probs_b = np.zeros((k, Hq, L), dtype=np.float64)
        for h in range(Hq):
            hk = h // g
            Kh = keys[b][:, hk, :]          # L x D
            Vh = vals[b][:, hk, :]          # L x D
            for j in range(k):
                visible = L - k + j + 1     # number of keys row j may read
                if visible <= 0:
                    continue
                s = scale * (Kh[:visible] @ q[b, j, h])
                m = np.max(s)
                e = np.exp(s - m)
                z = np.sum(e)
                p = e / z
                out[b, j, h] = p @ Vh[:visible]
                lse[b, j, h] = m + np.log(z)
                probs_b[j, h, :visible] = p
        all_probs.append(probs_b)
    if return_probs:
        return out, lse, all_probs
    return out, lse


def merge_partials(outs, lses):
    """Combine attention results over disjoint key subsets into the whole.

    Given per-subset normalised outputs o_i and log-sum-exps lse_i of the
    same query rows, the attention over the union of the subsets is
        lse = log sum_i exp(lse_i),  o = sum_i exp(lse_i - lse) o_i.
    Subsets with lse_i = -inf (no keys) contribute nothing.
    outs: [S, ..., D]; lses: [S, ...].  Returns (o, lse).
    """
    outs = np.asarray(outs, dtype=np.float64)
    lses = np.asarray(lses, dtype=np.float64)
    m = np.max(lses, axis=0)
    safe_m = np.where(np.isfinite(m), m, 0.0)
    w = np.exp(lses - safe_m[None])
    z = np.sum(w, axis=0)
    lse = np.where(z > 0, safe_m + np.log(np.where(z > 0, z, 1.0)), -np.inf)
    o = np.sum(w[..., None] * outs, axis=0) / np.where(z > 0, z, 1.0)[..., None]
    return o, lse
