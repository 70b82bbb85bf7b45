"""GPU parity of sd_latent_compress against the oracle (same seeded inputs)."""

import math

import numpy as np
import pytest

import oracle
from paper_2505_12728_amd import synth
from tests.gpu_util import assert_close, to_device

pytestmark = pytest.mark.gpu


def run_gpu(lat, feats, H, scale):
    import torch
    import paper_2505_12728_amd as sd
    out = sd.sd_latent_compress(to_device(lat), to_device(feats), H, scale)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def oracle_head(lat, feats, H, b, h, scale):
    dh = lat.shape[1] // H
    cols = slice(h * dh, (h + 1) * dh)
    return oracle.latent_compress(lat.values[:, cols], feats.values[b:b + 1, :, cols], 1, scale)


@pytest.mark.parametrize("wi", [0, 1, 2])
def test_compress_workload_full_oracle(wi):
    w = synth.workload(wi)
    print(f"compress workload {w.name}", flush=True)
    lat, feats = synth.compress_inputs(w)
    out = run_gpu(lat, feats, w.c_heads, 1.0)
    ref = oracle.latent_compress(lat.values, feats.values, w.c_heads, 1.0)
    assert_close(out, ref, w.dtype, w.name)


@pytest.mark.parametrize("wi", [3, 4])
def test_compress_workload_every_element(wi):
    # batched-paged (16 sequences) and long-video (4 x 16384 tokens, 64
    # heads, eight-wave groups) at full size: every (sequence, head) output
    # is compared with the oracle
    w = synth.workload(wi)
    print(f"compress workload {w.name}", flush=True)
    lat, feats = synth.compress_inputs(w)
    out = run_gpu(lat, feats, w.c_heads, 1.0)
    dh = w.c_width // w.c_heads
    ref = np.empty(out.shape)
    for b in range(w.c_batch):
        for h in range(w.c_heads):
            ref[b:b + 1, :, h * dh:(h + 1) * dh] = oracle_head(lat, feats, w.c_heads, b, h, 1.0)
    assert_close(out, ref, w.dtype, w.name)


CASES = [
    # name, dtype, B, N, C, d, H, scale
    ("ragged-tokens", "bf16", 2, 1000, 64, 256, 2, 1.0),
    ("latents-not-multiple", "bf16", 1, 777, 70, 256, 2, 1.0),
    ("diffuse-scale", "bf16", 1, 2048, 128, 512, 4, 1 / math.sqrt(128)),
    ("head-dim-64", "bf16", 2, 600, 96, 256, 4, 1 / 8),
    ("one-token", "bf16", 1, 1, 32, 128, 1, 1.0),
    ("many-latents", "bf16", 1, 300, 520, 128, 1, 1.0),
    ("split-tokens", "bf16", 1, 20000, 64, 128, 1, 1 / math.sqrt(128)),
    ("eight-waves-ragged-splits", "bf16", 1, 20037, 260, 256, 2, 1 / math.sqrt(128)),
    ("eight-waves-head-dim-64", "bf16", 1, 1500, 300, 128, 2, 1 / 8),
    # a negative scale is folded into the queries (bf16 sign flips on the
    # channel-major path of eight-wave groups, fp16 ones elsewhere); a zero
    # scale gives every token the same weight
    ("eight-waves-negative-scale", "bf16", 1, 3000, 256, 256, 2, -1 / math.sqrt(128)),
    ("four-waves-negative-scale", "bf16", 2, 900, 128, 256, 2, -0.5),
    ("eight-waves-zero-scale", "bf16", 1, 700, 256, 256, 2, 0.0),
    ("bf16-dh256", "bf16", 2, 700, 40, 512, 2, 1 / 16),
    ("bf16-dh256-one-token", "bf16", 1, 1, 9, 256, 1, 1.0),
    ("bf16-dh256-ragged", "bf16", 1, 3001, 17, 768, 3, 1 / 16),
    ("f32-heads", "f32", 2, 333, 20, 256, 2, 0.5),
    ("f32-dh256", "f32", 1, 2000, 16, 256, 1, 1 / 16),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_compress_edge_cases(case):
    name, dt, B, N, C, d, H, scale = case
    print(f"compress case {name}", flush=True)
    w = synth.Workload(name, dt, batch=1, hq=1, hkv=1, head_dim=64, kv_len=1, block=1,
                       c_batch=B, c_tokens=N, c_width=d, c_latents=C, c_heads=H)
    lat, feats = synth.compress_inputs(w, seed=17)
    out = run_gpu(lat, feats, H, scale)
    ref = oracle.latent_compress(lat.values, feats.values, H, scale)
    assert_close(out, ref, dt, name)


GRID_CASES = [
    # more (sequence, head) pairs, and more 64-token splits, than a grid's
    # y / z extent (65535) holds: the float64 kernel takes the rest in
    # grid-stride loops
    ("many-sequences", "f32", 70000, 3, 8, 64, 1),
    ("many-splits", "f32", 1, 65536 * 64 + 100, 8, 64, 1),
]


@pytest.mark.parametrize("case", GRID_CASES, ids=[c[0] for c in GRID_CASES])
def test_compress_beyond_grid_extent(case):
    name, dt, B, N, C, d, H = case
    print(f"compress grid case {name}", flush=True)
    w = synth.Workload(name, dt, batch=1, hq=1, hkv=1, head_dim=64, kv_len=1, block=1,
                       c_batch=B, c_tokens=N, c_width=d, c_latents=C, c_heads=H)
    lat, feats = synth.compress_inputs(w, seed=31)
    out = run_gpu(lat, feats, H, 1 / 8)
    ref = oracle.latent_compress(lat.values, feats.values, H, 1 / 8)
    assert_close(out, ref, dt, name)


RANGE_CASES = [
    # name, B, N, C, d, H, scale, what
    ("large-feats-8w", 1, 3000, 256, 256, 2, 1 / 64, "large"),       # eight-wave groups, token splits
    ("large-feats-4w", 2, 1000, 128, 256, 2, 1 / 64, "large"),
    ("tiny-feats", 1, 2000, 256, 256, 2, 1.0, "tiny"),
    ("tiny-feats-2w", 2, 700, 64, 256, 2, 1.0, "tiny"),
    ("large-latents", 1, 1500, 256, 256, 2, 1e-6, "large-latents"),
    ("mixed-subnormal", 1, 1200, 256, 256, 2, 1.0, "mixed"),
]


@pytest.mark.parametrize("case", RANGE_CASES, ids=[c[0] for c in RANGE_CASES])
def test_compress_outside_fp16_range(case):
    # bf16 values that fp16 does not hold exactly: magnitudes up to 1e5
    # (above 65280), a tensor scaled to ~1e-6 (every value below 2^-14, most
    # below fp16's subnormal resolution), latents above 65280, and a normal
    # tensor with a tenth of its values below 2^-14; all within the float
    # tolerance of the oracle on the same bf16 values
    name, B, N, C, d, H, scale, what = case
    print(f"compress range case {name}", flush=True)
    w = synth.Workload(name, "bf16", batch=1, hq=1, hkv=1, head_dim=64, kv_len=1, block=1,
                       c_batch=B, c_tokens=N, c_width=d, c_latents=C, c_heads=H)
    lat, feats = synth.compress_inputs(w, seed=23)
    rng = np.random.default_rng(29)
    F = feats.values.astype(np.float32).copy()
    Q = lat.values.astype(np.float32).copy()
    if what == "large":
        F *= np.float32(2000.0)                      # |F| up to ~1e4 everywhere
        idx = rng.integers(0, F.size, size=F.size // 50)
        F.reshape(-1)[idx] = rng.choice([-1.0, 1.0], size=idx.size).astype(np.float32) * \
            rng.uniform(65536.0, 1e5, size=idx.size).astype(np.float32)
    elif what == "tiny":
        F *= np.float32(1e-6)
    elif what == "large-latents":
        Q *= np.float32(3e4)
        Q.reshape(-1)[rng.integers(0, Q.size, size=Q.size // 20)] = np.float32(9e4)
    elif what == "mixed":
        idx = rng.integers(0, F.size, size=F.size // 10)
        F.reshape(-1)[idx] *= np.float32(2.0 ** -20)
    feats = synth.Tensor(F, "bf16")
    lat = synth.Tensor(Q, "bf16")
    if what == "large":
        assert np.abs(feats.values).max() > 65280
    out = run_gpu(lat, feats, H, scale)
    ref = oracle.latent_compress(lat.values, feats.values, H, scale)
    assert_close(out, ref, "bf16", name)


def test_compress_zero_queries_is_average_pooling_on_gpu():
    w = synth.Workload("pool", "bf16", batch=1, hq=1, hkv=1, head_dim=64, kv_len=1, block=1,
                       c_batch=2, c_tokens=500, c_width=256, c_latents=64, c_heads=2)
    lat, feats = synth.compress_inputs(w, seed=2)
    zero = synth.Tensor(np.zeros_like(lat.values), "bf16")
    out = run_gpu(zero, feats, 2, 1.0)
    mean = feats.values.astype(np.float64).mean(axis=1)
    assert_close(out, np.broadcast_to(mean[:, None, :], out.shape), "bf16", "pooling")


def test_compress_is_deterministic():
    w = synth.workload(2)
    lat, feats = synth.compress_inputs(w)
    a = run_gpu(lat, feats, w.c_heads, 1.0)
    b = run_gpu(lat, feats, w.c_heads, 1.0)
    assert np.array_equal(a, b)
