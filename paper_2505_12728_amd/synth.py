"""Seeded synthetic workloads for the draft-verify hot path.

This module only draws inputs: it holds none of the method's arithmetic
(no compression, attention or acceptance).  Both the HIP path and the CPU
oracle are fed from it, so the two always see the same bytes.

The paper's workloads (Kinetics-400 video captioning and LLaVA-instruct
visual instruction tuning, Sec. 4.1) are not available; seeded tensors with
the shapes of its image and video settings stand in for them:

* features, latents, queries, keys and values ~ N(0, 1), drawn in float32
  and, for bfloat16 workloads, rounded once to bfloat16 (round to nearest
  even); both sides consume the rounded values;
* target logits ~ N(0, 3^2) of shape [B, k+1, V]; draft logits are the
  first k target rows plus N(0, 1) noise; p = softmax(z / tau) and
  q = softmax(z' / tau) are formed in float64 and stored as float32 once;
* drafted ids: in sampled mode x_i ~ q_i (float64 inverse CDF on a
  separate stream), in greedy mode x_i = argmax q_i;
* acceptance uniforms on the 2^-24 grid, one stream per sequence;
* paged caches: per-sequence lengths uniform in a range, 16-token pages
  with a random page permutation, padding slots and spare pages poisoned.

Every tensor has its own Philox streams keyed by (seed, tensor, chunk), so
changing one size does not change the other tensors' values, and large
tensors are drawn in parallel threads without changing any value.
"""

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

BASE_SEED = 2505_12728
PAGE_SIZE = 16
POISON = 8192.0          # exact in bfloat16 and float32

# stream order for SeedSequence.spawn; never reorder (it changes every value)
_STREAMS = ("latents", "feats", "q", "k", "v", "target_logits", "draft_noise",
            "draft_uniforms", "accept_uniforms", "kv_lens", "page_perm",
            "lm_hidden", "lm_weight", "sample_uniforms", "draft_u", "draft_w",
            "draft_cache")


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shapes of one synthetic workload (all three operations)."""
    name: str
    dtype: str                  # "f32" or "bf16"
    # verification attention
    batch: int
    hq: int
    hkv: int
    head_dim: int
    kv_len: int                 # contiguous length, or the upper bound when paged
    block: int                  # k drafted tokens verified in one pass
    paged: bool = False
    kv_len_min: int = 0         # paged workloads draw lengths in [kv_len_min, kv_len]
    # latent compression (Eq. 3)
    c_batch: int = 1
    c_tokens: int = 0           # N visual tokens
    c_width: int = 0            # d
    c_latents: int = 0          # C learned queries
    c_heads: int = 1
    # acceptance
    vocab: int = 0
    modes: tuple = ("sampled",)
    temperature: float = 1.0
    # LM head (hidden width d of the head; its rows are the batch's k+1
    # target positions)
    lm_width: int = 0
    # draft semi-AR layer: the target layer's heads and width (d = hq *
    # head_dim), MLP width I, cached context length before the step (the
    # compressed visual rows plus earlier text); the step's rows per
    # sequence are one accepted token and the k placeholders
    draft_ffn: int = 0
    draft_ctx: int = 0

    @property
    def seed(self):
        return BASE_SEED + WORKLOADS.index(self)


WORKLOADS = [
    Workload("tiny-f32", "f32", batch=1, hq=4, hkv=1, head_dim=64, kv_len=608,
             block=4, c_batch=1, c_tokens=576, c_width=256, c_latents=16,
             c_heads=1, vocab=1024, modes=("sampled", "greedy"),
             temperature=1.0, lm_width=256, draft_ffn=512, draft_ctx=24),
    Workload("llava-7b-image", "bf16", batch=1, hq=32, hkv=32, head_dim=128,
             kv_len=1200, block=5, c_batch=1, c_tokens=576, c_width=4096,
             c_latents=64, c_heads=32, vocab=32000, modes=("sampled",),
             temperature=1.0, lm_width=4096, draft_ffn=11008, draft_ctx=96),
    Workload("qwen2vl-7b-video", "bf16", batch=1, hq=28, hkv=4, head_dim=128,
             kv_len=6528, block=8, c_batch=1, c_tokens=6272, c_width=3584,
             c_latents=256, c_heads=28, vocab=152064,
             modes=("greedy", "sampled"), temperature=1.0, lm_width=3584,
             draft_ffn=18944, draft_ctx=288),
    Workload("batched-paged", "bf16", batch=16, hq=32, hkv=8, head_dim=128,
             kv_len=16384, kv_len_min=2048, block=6, paged=True, c_batch=16,
             c_tokens=1024, c_width=4096, c_latents=128, c_heads=32,
             vocab=32000, modes=("sampled",), temperature=1.0, lm_width=4096,
             draft_ffn=14336, draft_ctx=160),
    Workload("long-video", "bf16", batch=4, hq=64, hkv=8, head_dim=128,
             kv_len=65536, block=8, c_batch=4, c_tokens=16384, c_width=8192,
             c_latents=512, c_heads=64, vocab=152064, modes=("sampled",),
             temperature=0.7, lm_width=8192, draft_ffn=28672, draft_ctx=544),
]


def workload(index_or_name):
    if isinstance(index_or_name, int):
        return WORKLOADS[index_or_name]
    for w in WORKLOADS:
        if w.name == index_or_name:
            return w
    raise KeyError(index_or_name)


# ---------------------------------------------------------------- helpers

_THREADS = max(1, min(16, os.cpu_count() or 1))
_CHUNK = 1 << 22


class Stream:
    """A named, seeded source of random draws.

    Scalar-sized draws come from one Philox generator keyed by
    (seed, stream index); large normal tensors are cut into 2^22-element
    chunks, each with its own Philox generator keyed by (seed, stream index,
    chunk index), and filled in parallel threads.  The values depend only on
    the seed, the stream and the shape, never on the thread count.
    """

    def __init__(self, seed, index):
        self.seed = seed
        self.index = index
        self.gen = np.random.Generator(np.random.Philox(
            np.random.SeedSequence(seed, spawn_key=(index,))))
        self._calls = 0

    def normal(self, shape):
        """N(0, 1) float32 draws of the given shape."""
        call = self._calls
        self._calls += 1
        total = int(np.prod(shape))
        out = np.empty(total, dtype=np.float32)

        def fill(job):
            ci, s = job
            g = np.random.Generator(np.random.Philox(
                np.random.SeedSequence(self.seed, spawn_key=(self.index, call, ci))))
            g.standard_normal(min(total, s + _CHUNK) - s, dtype=np.float32,
                              out=out[s:min(total, s + _CHUNK)])

        jobs = list(enumerate(range(0, total, _CHUNK)))
        if len(jobs) > 1 and _THREADS > 1:
            with ThreadPoolExecutor(_THREADS) as ex:
                list(ex.map(fill, jobs))
        else:
            for j in jobs:
                fill(j)
        return out.reshape(shape)


def streams(seed):
    """One independent stream per named tensor."""
    return {name: Stream(seed, i) for i, name in enumerate(_STREAMS)}


def _parallel_map(fn, x, out):
    """Apply an elementwise numpy function chunk by chunk in threads."""
    xf = x.reshape(-1)
    of = out.reshape(-1)
    jobs = range(0, xf.size, _CHUNK)

    def run(s):
        of[s:s + _CHUNK] = fn(xf[s:s + _CHUNK])

    if xf.size > _CHUNK and _THREADS > 1:
        with ThreadPoolExecutor(_THREADS) as ex:
            list(ex.map(run, jobs))
    else:
        for s in jobs:
            run(s)
    return out


def _bf16_round(x):
    bits = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((bits >> np.uint32(16)) & np.uint32(1))
    return ((bits + bias) >> np.uint32(16)).astype(np.uint16)


def _bf16_widen(bits):
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def bf16_bits(x):
    """Round float32 values to bfloat16 (nearest even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return _parallel_map(_bf16_round, x, np.empty(x.shape, np.uint16))


def bf16_to_f32(bits):
    """Widen bfloat16 bit patterns to the float32 values they denote."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return _parallel_map(_bf16_widen, bits, np.empty(bits.shape, np.float32))


class Tensor:
    """A host tensor as both sides see it.

    ``values`` holds the exact float32 values (already bfloat16-rounded for
    bf16 tensors); ``bits`` holds the uint16 storage for bf16 tensors.
    """

    def __init__(self, values, dtype):
        self.dtype = dtype
        if dtype == "bf16":
            self.bits = bf16_bits(values)
            self.values = bf16_to_f32(self.bits)
        elif dtype == "f32":
            self.bits = None
            self.values = np.ascontiguousarray(values, dtype=np.float32)
        else:
            raise ValueError(dtype)

    @property
    def shape(self):
        return self.values.shape


def normal(stream, shape):
    return stream.normal(shape)


# ------------------------------------------------------ per-operation inputs

def compress_inputs(w, seed=None, batch=None, tokens=None):
    """Learned queries [C, d] and visual features [B, N, d] for Eq. 3."""
    rs = streams(w.seed if seed is None else seed)
    B = w.c_batch if batch is None else batch
    N = w.c_tokens if tokens is None else tokens
    latents = Tensor(normal(rs["latents"], (w.c_latents, w.c_width)), w.dtype)
    feats = Tensor(normal(rs["feats"], (B, N, w.c_width)), w.dtype)
    return latents, feats


Q8_EXP_MIN, Q8_EXP_MAX = -14, 9    # every q * 2^e (|q| <= 127) a normal fp16 or zero


def quantize_pow2_rows(x):
    """int8 rows with one power-of-two scale each (the int8 compressor's
    input format): e = ceil(log2(max|row| / 127)) clamped to [-14, 9],
    q = clip(round(x / 2^e), -127, 127).  Returns (q int8, e int8)."""
    x = np.asarray(x, dtype=np.float32)
    amax = np.max(np.abs(x), axis=-1)
    with np.errstate(divide="ignore"):
        e = np.ceil(np.log2(np.maximum(amax, 1e-30) / 127.0))
    e = np.clip(e, Q8_EXP_MIN, Q8_EXP_MAX).astype(np.int8)
    q = np.empty(x.shape, dtype=np.int8)
    scale = np.exp2(-e.astype(np.float32))[..., None]
    q[...] = np.clip(np.rint(x * scale), -127, 127)
    return q, e


def compress_q8_inputs(w, seed=None, batch=None, tokens=None):
    """The compression inputs of ``compress_inputs`` quantised to int8 rows
    with power-of-two scales: latents_q [C, d], latent_exp [C], feats_q
    [B, N, d], feat_exp [B, N] (int8 each)."""
    lat, feats = compress_inputs(w, seed, batch, tokens)
    lq, le = quantize_pow2_rows(lat.values)
    fq, fe = quantize_pow2_rows(feats.values)
    return {"latents_q": lq, "latent_exp": le, "feats_q": fq, "feat_exp": fe}


def compress_q8_bytes(w):
    """F_V's int8 rows and exponents once, the latents' likewise, the fp32
    output once."""
    return (w.c_batch * w.c_tokens * (w.c_width + 1) + w.c_latents * (w.c_width + 1)
            + w.c_batch * w.c_latents * w.c_width * 4)


def kv_lengths(w, seed=None):
    rs = streams(w.seed if seed is None else seed)
    if not w.paged:
        return np.full(w.batch, w.kv_len, dtype=np.int32)
    return rs["kv_lens"].gen.integers(w.kv_len_min, w.kv_len + 1,
                                  size=w.batch).astype(np.int32)


def verify_inputs(w, seed=None, kv_len=None, poison=POISON):
    """Queries, KV cache (contiguous or paged) and lengths for verification.

    Returns a dict with q [B, k, Hq, D]; k_cache / v_cache as
    [B, Lmax, Hkv, D] (contiguous) or [P, Hkv, 16, D] page pools; kv_len [B];
    page_table [B, max_pages] int32 or None.  Cache slots that no sequence
    owns (padding, spare pages) hold ``poison``.
    """
    seed = w.seed if seed is None else seed
    rs = streams(seed)
    lens = kv_lengths(w, seed) if kv_len is None else np.asarray(kv_len, np.int32)
    B, k, Hq, Hkv, D = w.batch, w.block, w.hq, w.hkv, w.head_dim
    q = Tensor(normal(rs["q"], (B, k, Hq, D)), w.dtype)
    if not w.paged:
        Lmax = int(max(w.kv_len, int(lens.max()) if lens.size else 0))
        kf = normal(rs["k"], (B, Lmax, Hkv, D))
        vf = normal(rs["v"], (B, Lmax, Hkv, D))
        for b in range(B):
            kf[b, lens[b]:] = poison
            vf[b, lens[b]:] = poison
        return {"q": q, "k_cache": Tensor(kf, w.dtype), "v_cache": Tensor(vf, w.dtype),
                "kv_len": lens, "page_table": None, "max_pages": 0, "lmax": Lmax}
    pages = [int(math.ceil(int(L) / PAGE_SIZE)) for L in lens]
    max_pages = max(1, int(math.ceil(w.kv_len / PAGE_SIZE)))
    n_pool = sum(pages) + 64
    perm = rs["page_perm"].gen.permutation(n_pool).astype(np.int32)
    page_table = np.zeros((B, max_pages), dtype=np.int32)
    pos = 0
    for b in range(B):
        page_table[b, :pages[b]] = perm[pos:pos + pages[b]]
        # entries past the sequence's last page point at a spare page; they
        # are never read for valid keys
        page_table[b, pages[b]:] = perm[-1]
        pos += pages[b]
    kf = np.full((n_pool, Hkv, PAGE_SIZE, D), poison, dtype=np.float32)
    vf = np.full((n_pool, Hkv, PAGE_SIZE, D), poison, dtype=np.float32)
    kg = rs["k"]
    vg = rs["v"]
    for b in range(B):
        L = int(lens[b])
        kl = normal(kg, (L, Hkv, D))          # the sequence's logical cache
        vl = normal(vg, (L, Hkv, D))
        for i in range(pages[b]):
            valid = min(PAGE_SIZE, L - i * PAGE_SIZE)
            pg = page_table[b, i]
            kf[pg, :, :valid] = kl[i * PAGE_SIZE:i * PAGE_SIZE + valid].transpose(1, 0, 2)
            vf[pg, :, :valid] = vl[i * PAGE_SIZE:i * PAGE_SIZE + valid].transpose(1, 0, 2)
    return {"q": q, "k_cache": Tensor(kf, w.dtype), "v_cache": Tensor(vf, w.dtype),
            "kv_len": lens, "page_table": page_table, "max_pages": max_pages,
            "lmax": 0}


def _probs(z, tau):
    """softmax(z / tau) along the last axis in float64, stored as float32."""
    z = np.asarray(z, dtype=np.float64) / tau
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return (e / e.sum(axis=-1, keepdims=True)).astype(np.float32)


def _accept_draws(w, mode, seed, batch):
    """Target / draft logits (float64), temperature and drafted ids."""
    rs = streams(w.seed if seed is None else seed)
    B = w.batch if batch is None else batch
    k, V = w.block, w.vocab
    tau = w.temperature if mode == "sampled" else 1.0
    z = 3.0 * normal(rs["target_logits"], (B, k + 1, V)).astype(np.float64)
    zd = z[:, :k] + normal(rs["draft_noise"], (B, k, V)).astype(np.float64)
    q = _probs(zd, tau)
    if mode == "greedy":
        draft = np.argmax(q, axis=-1).astype(np.int32)
    else:
        draft = np.empty((B, k), dtype=np.int32)
        du = rs["draft_uniforms"].gen.random((B, k))
        for b in range(B):
            for i in range(k):
                c = np.cumsum(q[b, i].astype(np.float64))
                draft[b, i] = min(V - 1, int(np.searchsorted(c, du[b, i] * c[-1],
                                                             side="right")))
    return z, zd, q, tau, draft


def accept_inputs(w, mode, seed=None, batch=None):
    """Target / draft probabilities, drafted ids and uniforms.

    Returns a dict with p [B, k+1, V] float32, q [B, k, V] float32,
    draft [B, k] int32 and u [B, k+1] float32 (multiples of 2^-24).
    """
    z, _, q, tau, draft = _accept_draws(w, mode, seed, batch)
    B, k = draft.shape
    p = _probs(z, tau)
    # one independent uniform stream per sequence
    base = w.seed if seed is None else seed
    ui = _STREAMS.index("accept_uniforms")
    u = np.empty((B, k + 1), dtype=np.float32)
    for b in range(B):
        g = np.random.Generator(np.random.Philox(
            np.random.SeedSequence(base, spawn_key=(ui, 1 << 20, b))))
        u[b] = (g.integers(0, 1 << 24, size=k + 1).astype(np.float64)
                * 2.0 ** -24).astype(np.float32)
    return {"p": p, "q": q, "draft": draft, "u": u, "temperature": tau}


def accept_logits_inputs(w, mode, seed=None, batch=None):
    """The same draws handed over as logits: target_logits [B, k+1, V] and
    draft_logits [B, k, V] (float32), draft [B, k] int32, the temperature and
    a key / offset for the device-side uniforms."""
    z, zd, _, tau, draft = _accept_draws(w, mode, seed, batch)
    base = w.seed if seed is None else seed
    return {"target_logits": z.astype(np.float32), "draft_logits": zd.astype(np.float32),
            "draft": draft, "temperature": tau,
            "philox_seed": (0x5EED0000 + 7919 * base) & ((1 << 64) - 1), "philox_offset": 3}


# --------------------------------------------------------- byte / flop counts

def lm_inputs(w, seed=None, rows=None, vocab=None):
    """LM head inputs: hidden states [R, d] ~ N(0, 1) and a head weight
    [V, d] ~ N(0, 9 / d) (logits then spread like N(0, 3^2), as the
    synthetic target logits do), in the workload's dtype, plus R sampling
    uniforms on the 2^-24 grid.  R defaults to batch * (k + 1)."""
    rs = streams(w.seed if seed is None else seed)
    R = w.batch * (w.block + 1) if rows is None else rows
    V = w.vocab if vocab is None else vocab
    d = w.lm_width
    hidden = Tensor(normal(rs["lm_hidden"], (R, d)), w.dtype)
    wv = normal(rs["lm_weight"], (V, d))
    _parallel_map(lambda x: x * np.float32(3.0 / math.sqrt(d)), wv, wv)
    weight = Tensor(wv, w.dtype)
    del wv
    u = (rs["sample_uniforms"].gen.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    return {"hidden": hidden, "weight": weight, "u": u, "temperature": w.temperature}


def lm_bytes(w, rows=None):
    """Algorithmic HBM bytes of one LM head pass: the weight and the hidden
    states read once, the probabilities written once."""
    R = w.batch * (w.block + 1) if rows is None else rows
    es = 2 if w.dtype == "bf16" else 4
    return w.vocab * w.lm_width * es + R * w.lm_width * es + R * w.vocab * 4


def verify_kv_bytes(w, lens=None):
    """K and V bytes the verification must read once: 2 * Hkv * D * es per token."""
    es = 4 if w.dtype == "f32" else 2
    lens = kv_lengths(w) if lens is None else lens
    return int(np.sum(lens, dtype=np.int64)) * 2 * w.hkv * w.head_dim * es


def compress_flops(w):
    """4 * d_h flops per (latent, token, head): 4 * B * C * N * d in total."""
    return 4 * w.c_batch * w.c_latents * w.c_tokens * w.c_width


def compress_bytes(w):
    es = 4 if w.dtype == "f32" else 2
    return (w.c_batch * w.c_tokens * w.c_width * es + w.c_latents * w.c_width * es
            + w.c_batch * w.c_latents * w.c_width * 4)


DRAFT_EPS = 1e-6
DRAFT_THETA = 10000.0


def draft_dims(w):
    """(B, r, d, hq, hkv, I, Lmax) of the workload's draft step."""
    d = w.hq * w.head_dim
    r = w.block + 1
    Lmax = (w.draft_ctx + 3 * (w.batch - 1) + r + 15) // 16 * 16 + 16
    return w.batch, r, d, w.hq, w.hkv, w.draft_ffn, Lmax


def draft_inputs(w, seed=None, batch=None, q8=False):
    """Inputs of one draft step, always in bfloat16 (weights, u, caches):
    u = concat(F_T, E) ~ N(0, 1) of shape [B, r, 2d]; projection weights
    ~ N(0, 1 / fan_in), so every projection maps unit-variance rows to
    unit-variance rows; RMSNorm weights 1 + N(0, 0.1^2) and the FC bias
    N(0, 0.1^2) in float32; the caches hold N(0, 1) context keys and values
    at positions 0 .. pos[b] - 1 and the poison value elsewhere; pos[b] =
    draft_ctx + 3 b (ragged contexts).  With q8, every projection is int8
    rows wq = clip(round(40 z), -127, 127), z ~ N(0, 1), under its name and
    float32 row scales 1 / (40 sqrt(fan_in)) under name + "_s" (the same
    N(0, 1 / fan_in) spread)."""
    rs = streams(w.seed if seed is None else seed)
    B, r, d, hq, hkv, I, Lmax = draft_dims(w)
    B = B if batch is None else batch
    D = d // hq

    weights_q8 = {}

    def weight(shape, fan_in):
        x = normal(rs["draft_w"], shape)
        if q8:
            _parallel_map(lambda v: np.clip(np.rint(v * np.float32(40.0)), -127, 127), x, x)
            wq = x.astype(np.int8)
            del x
            return wq, np.full(shape[0], 1.0 / (40.0 * math.sqrt(fan_in)), dtype=np.float32)
        _parallel_map(lambda v: v * np.float32(1.0 / math.sqrt(fan_in)), x, x)
        t = Tensor(x, "bf16")
        del x
        return t

    u = Tensor(normal(rs["draft_u"], (B, r, 2 * d)), "bf16")
    W = {"fc_w": weight((d, 2 * d), 2 * d),
         "fc_b": (normal(rs["draft_w"], (d,)) * np.float32(0.1)).astype(np.float32),
         "ln1": (1.0 + normal(rs["draft_w"], (d,)) * np.float32(0.1)).astype(np.float32),
         "wqkv": weight(((hq + 2 * hkv) * D, d), d),
         "wo": weight((d, hq * D), hq * D),
         "ln2": (1.0 + normal(rs["draft_w"], (d,)) * np.float32(0.1)).astype(np.float32),
         "wgu": weight((2 * I, d), d),
         "wdown": weight((d, I), I)}
    if q8:
        for name in ("fc_w", "wqkv", "wo", "wgu", "wdown"):
            W[name], W[name + "_s"] = W[name]
    pos = (w.draft_ctx + 3 * np.arange(B)).astype(np.int32)
    kc = normal(rs["draft_cache"], (B, Lmax, hkv, D))
    vc = normal(rs["draft_cache"], (B, Lmax, hkv, D))
    for b in range(B):
        kc[b, pos[b]:] = POISON
        vc[b, pos[b]:] = POISON
    return {"u": u, "weights": W, "k_cache": Tensor(kc, "bf16"), "v_cache": Tensor(vc, "bf16"),
            "pos": pos, "eps": DRAFT_EPS, "theta": DRAFT_THETA, "hq": hq, "hkv": hkv}


def draft_bytes(w):
    """Algorithmic HBM bytes of one draft step: every weight once (bf16),
    the rows' input and output, and the cache entries the attention reads
    (keys and values of positions 0 .. pos[b] + r - 1) and writes."""
    B, r, d, hq, hkv, I, Lmax = draft_dims(w)
    D = d // hq
    params = d * 2 * d + (hq + 2 * hkv) * D * d + d * hq * D + 2 * I * d + d * I
    ctx = sum(w.draft_ctx + 3 * b + r for b in range(B))
    return 2 * params + B * r * (2 * d * 2 + d * 4) + ctx * 2 * hkv * D * 2


def draft_kp_bytes(w, kp):
    """Algorithmic HBM bytes of K = block drafts in K / kp passes: per pass
    the draft layer's weights once (and its rows and cache traffic), the
    LM head weight once and the kp rows' distributions written once."""
    B, r, d, hq, hkv, I, Lmax = draft_dims(w)
    D = d // hq
    passes = w.block // kp
    params = d * 2 * d + (hq + 2 * hkv) * D * d + d * hq * D + 2 * I * d + d * I
    per_pass = 2 * params + 2 * w.vocab * d + B * kp * w.vocab * 4
    ctx = sum(w.draft_ctx + 3 * b + r for b in range(B))
    return passes * per_pass + ctx * 2 * hkv * D * 2


def draft_q8_bytes(w):
    """Algorithmic HBM bytes of one int8 draft step: every int8 weight once
    and its row scales, plus the rows and cache traffic of draft_bytes."""
    B, r, d, hq, hkv, I, Lmax = draft_dims(w)
    D = d // hq
    params = d * 2 * d + (hq + 2 * hkv) * D * d + d * hq * D + 2 * I * d + d * I
    rows = d + (hq + 2 * hkv) * D + d + 2 * I + d
    return draft_bytes(w) - 2 * params + params + 4 * rows
