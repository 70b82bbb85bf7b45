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
