"""GPU parity of sd_latent_compress_q8 (the int8 draft's compressor: int8
rows with power-of-two row scales) against the oracle on the same int8
values, within the bf16 float tolerance."""

import math

import numpy as np
import pytest

import oracle
from paper_2505_12728_amd import synth
from tests.gpu_util import assert_close, np_to_device

pytestmark = pytest.mark.gpu


def run_gpu(q, H, scale):
    import torch
    import paper_2505_12728_amd as sd
    out = sd.sd_latent_compress_q8(np_to_device(q["latents_q"]), np_to_device(q["latent_exp"]),
                                   np_to_device(q["feats_q"]), np_to_device(q["feat_exp"]), H, scale)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def oracle_full(q, H, scale):
    """Oracle output assembled per (sequence, head) slice (bounded memory)."""
    lq, le, fq, fe = q["latents_q"], q["latent_exp"], q["feats_q"], q["feat_exp"]
    C, d = lq.shape
    B = fq.shape[0]
    dh = d // H
    ref = np.empty((B, C, d))
    for b in range(B):
        for h in range(H):
            cols = slice(h * dh, (h + 1) * dh)
            ref[b:b + 1, :, cols] = oracle.latent_compress_q8(lq[:, cols], le, fq[b:b + 1, :, cols],
                                                              fe[b:b + 1], 1, scale)
    return ref


@pytest.mark.parametrize("wi", [1, 2, 3, 4])
def test_compress_q8_workload_every_element(wi):
    # the four bf16 workloads' compression shapes (128-channel heads), every
    # output element
    w = synth.workload(wi)
    print(f"compress q8 workload {w.name}", flush=True)
    q = synth.compress_q8_inputs(w)
    out = run_gpu(q, w.c_heads, 1.0)
    assert_close(out, oracle_full(q, w.c_heads, 1.0), "bf16", w.name)


CASES = [
    # name, B, N, C, d, H, scale: one to eight waves per work-group, ragged
    # token and latent counts, token splits past the int8 split limit
    ("ragged-tokens", 2, 1000, 64, 256, 2, 1.0),
    ("latents-not-multiple", 1, 777, 70, 256, 2, 1.0),
    ("one-wave", 1, 300, 20, 128, 1, 1.0),
    ("diffuse-scale", 1, 2048, 128, 512, 4, 1 / math.sqrt(128)),
    ("one-token", 1, 1, 32, 128, 1, 1.0),
    ("eight-waves-splits", 1, 20037, 260, 256, 2, 1 / math.sqrt(128)),
    ("long-split", 1, 40000, 256, 128, 1, 1.0),
    ("eight-waves-negative-scale", 1, 3000, 256, 256, 2, -1 / math.sqrt(128)),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_compress_q8_edge_cases(case):
    name, B, N, C, d, H, scale = case
    print(f"compress q8 case {name}", flush=True)
    w = synth.Workload(name, "bf16", batch=1, hq=1, hkv=1, head_dim=64, kv_len=1, block=1,
                       c_batch=B, c_tokens=N, c_width=d, c_latents=C, c_heads=H)
    q = synth.compress_q8_inputs(w, seed=19)
    out = run_gpu(q, H, scale)
    assert_close(out, oracle_full(q, H, scale), "bf16", name)


def test_compress_q8_exponent_range_ends_and_zero_rows():
    # exponents at both ends of [-14, 9] on a mix of tokens, all-zero rows,
    # latents at the ends too; every value is exact in fp16
    rng = np.random.default_rng(41)
    B, N, C, d, H = 2, 700, 96, 256, 2
    lq = rng.integers(-127, 128, size=(C, d)).astype(np.int8)
    le = rng.choice([-14, -9, -6, 0, 2], size=C).astype(np.int8)
    fq = rng.integers(-127, 128, size=(B, N, d)).astype(np.int8)
    fe = rng.choice([-14, -12, -7, -6, -5, 3, 9], size=(B, N)).astype(np.int8)
    fq[:, 5] = 0
    fq[1, 100:110] = 0
    lq[7] = 0
    q = {"latents_q": lq, "latent_exp": le, "feats_q": fq, "feat_exp": fe}
    scale = 2.0 ** -12                          # scores of a usable spread
    out = run_gpu(q, H, scale)
    assert_close(out, oracle_full(q, H, scale), "bf16", "exponent ends")


def test_compress_q8_equals_bf16_path_on_pow2_exact_inputs():
    # int8 rows times powers of two are exact bf16 values too: the int8 and
    # bf16 entry points see the same numbers and must agree to rounding order
    import torch
    import paper_2505_12728_amd as sd
    w = synth.Workload("eq", "bf16", batch=1, hq=1, hkv=1, head_dim=64, kv_len=1, block=1,
                       c_batch=2, c_tokens=1500, c_width=256, c_latents=256, c_heads=2)
    q = synth.compress_q8_inputs(w, seed=5)
    lat = synth.Tensor(oracle.dequantize_pow2_rows(q["latents_q"], q["latent_exp"]).astype(np.float32), "bf16")
    feats = synth.Tensor(oracle.dequantize_pow2_rows(q["feats_q"], q["feat_exp"]).astype(np.float32), "bf16")
    to = lambda t: torch.from_numpy(np.ascontiguousarray(t.bits).view(np.int16)).view(torch.bfloat16).cuda()
    a = sd.sd_latent_compress(to(lat), to(feats), 2, 1.0).cpu().numpy()
    b = run_gpu(q, 2, 1.0)
    ref = oracle_full(q, 2, 1.0)
    assert_close(a, ref, "bf16", "bf16 path")
    assert_close(b, ref, "bf16", "int8 path")
    assert np.max(np.abs(a - b)) <= 1e-3 * np.sqrt(np.mean(ref * ref))


def test_compress_q8_is_deterministic():
    w = synth.workload(2)
    q = synth.compress_q8_inputs(w)
    assert np.array_equal(run_gpu(q, w.c_heads, 1.0), run_gpu(q, w.c_heads, 1.0))
