"""GPU parity of sd_lm_head_probs (within the float tolerance) and
sd_sample_tokens (bit-exact) against the oracle."""

import numpy as np
import pytest

import oracle
from paper_2505_12728_amd import synth
from tests.gpu_util import assert_probs_close, np_to_device, to_device

pytestmark = pytest.mark.gpu


def run_probs(hidden, weight, tau):
    import torch
    import paper_2505_12728_amd as sd
    p = sd.sd_lm_head_probs(to_device(hidden), to_device(weight), tau)
    torch.cuda.synchronize()
    return p.cpu().numpy()


def ref_probs(hidden, weight, tau, rows=None):
    """Oracle probabilities of the given rows, logits formed 8192 entries at
    a time (float64 per chunk) to bound host memory."""
    h = hidden.values if rows is None else hidden.values[rows]
    V = weight.shape[0]
    z = np.concatenate([oracle.lm_head_logits(h, weight.values[v:v + 8192])
                        for v in range(0, V, 8192)], axis=1)
    return oracle.softmax_temperature(z, tau), z


def check_probs(gpu, ref, z, dtype, what):
    assert_probs_close(gpu, ref, dtype, what)
    assert np.allclose(gpu.sum(axis=1), 1.0, atol=1e-4), f"{what}: rows do not sum to 1"
    if z.shape[1] < 2:
        return
    # the most likely entry agrees wherever the top two logits are apart
    top2 = np.sort(z, axis=1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) > 1e-3
    assert np.array_equal(np.argmax(gpu, axis=1)[clear], np.argmax(z, axis=1)[clear]), what


@pytest.mark.parametrize("name", ["tiny-f32", "llava-7b-image", "qwen2vl-7b-video", "batched-paged"])
def test_lm_head_workloads(name):
    w = synth.workload(name)
    inp = synth.lm_inputs(w)
    gpu = run_probs(inp["hidden"], inp["weight"], inp["temperature"])
    ref, z = ref_probs(inp["hidden"], inp["weight"], inp["temperature"])
    check_probs(gpu, ref, z, w.dtype, name)


def test_lm_head_long_video_every_row():
    # full size (36 rows, d 8192, V 152064, tau 0.7), every probability
    w = synth.workload("long-video")
    inp = synth.lm_inputs(w)
    gpu = run_probs(inp["hidden"], inp["weight"], inp["temperature"])
    ref, z = ref_probs(inp["hidden"], inp["weight"], inp["temperature"])
    check_probs(gpu, ref, z, "bf16", "long-video")


@pytest.mark.parametrize("R,d,V,tau", [(1, 64, 1, 1.0), (1, 64, 37, 0.5), (5, 128, 1000, 0.05),
                                       (17, 192, 300, 20.0), (65, 64, 129, 1.0),
                                       (130, 128, 2050, 0.7),
                                       # widths d % 256 == 0 with R <= 64 (the
                                       # 512-byte-run kernel): one entry, a
                                       # partial tile, an odd chunk count, the
                                       # largest row count, 8-wave tiles with a
                                       # ragged end and unaligned rows
                                       (1, 256, 1, 1.0), (3, 256, 50, 0.5),
                                       (16, 512, 1000, 1.0), (33, 768, 129, 2.0),
                                       (64, 256, 65600, 0.7), (49, 1024, 70001, 0.3)])
def test_lm_head_edge_shapes(R, d, V, tau):
    # ragged rows (row blocks of 16, launches of 64), ragged vocabulary
    # (tiles of 64 / 128, blocks of 16), odd channel groups, extreme
    # temperatures
    w = synth.workload("llava-7b-image")
    rs = synth.streams(1234 + R + V)
    hidden = synth.Tensor(rs["lm_hidden"].normal((R, d)), "bf16")
    weight = synth.Tensor(rs["lm_weight"].normal((V, d)) * np.float32(3.0 / np.sqrt(d)), "bf16")
    gpu = run_probs(hidden, weight, tau)
    ref, z = ref_probs(hidden, weight, tau)
    assert gpu.shape == (R, V)
    check_probs(gpu, ref, z, "bf16", f"R{R} d{d} V{V} tau{tau}")


def test_lm_head_fp32_matches_tightly():
    rs = synth.streams(77)
    hidden = synth.Tensor(rs["lm_hidden"].normal((9, 100)), "f32")
    weight = synth.Tensor(rs["lm_weight"].normal((515, 100)) * np.float32(0.3), "f32")
    gpu = run_probs(hidden, weight, 0.9)
    ref, z = ref_probs(hidden, weight, 0.9)
    assert_probs_close(gpu, ref, "f32", "fp32 head")


def test_lm_head_is_deterministic():
    w = synth.workload("llava-7b-image")
    inp = synth.lm_inputs(w, rows=20, vocab=5000)
    a = run_probs(inp["hidden"], inp["weight"], 1.0)
    b = run_probs(inp["hidden"], inp["weight"], 1.0)
    assert np.array_equal(a, b)


# ------------------------------------------------------------- sampling

def run_sample(probs, u):
    import torch
    import paper_2505_12728_amd as sd
    t = sd.sd_sample_tokens(np_to_device(np.ascontiguousarray(probs, np.float32)),
                            np_to_device(np.ascontiguousarray(u, np.float32)))
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.mark.parametrize("name", ["tiny-f32", "llava-7b-image", "qwen2vl-7b-video", "long-video"])
def test_sample_tokens_workloads(name):
    # distributions of the workload's shape from the oracle (float64,
    # stored as float32), drawn with the workload's uniforms: bit-exact
    w = synth.workload(name)
    R, V = w.batch * w.block, w.vocab
    rs = synth.streams(w.seed + 1000)
    z = rs["target_logits"].normal((R, V)).astype(np.float64) * 3.0
    probs = oracle.softmax_temperature(z, w.temperature).astype(np.float32)
    u = (rs["sample_uniforms"].gen.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)
    assert np.array_equal(run_sample(probs, u), oracle.sample_tokens(probs, u)), name


def test_sample_tokens_edge_cases():
    p = np.zeros((6, 300), dtype=np.float32)
    p[0, :4] = [0.25, 0.5, 0.125, 0.125]          # dyadic thresholds
    p[1, 299] = 1.0                              # last entry
    p[2, 5] = 1e-13                              # weights all zero: argmax
    p[2, 7] = 4e-13
    p[4, :] = 1.0 / 300                          # uniform
    p[5, 100:] = 2.0                             # values above 1 are clamped
    u = np.array([0.75, 0.0, 0.5, 0.3, 1 - 2 ** -24, 0.6], dtype=np.float32)
    got = run_sample(p, u)
    assert np.array_equal(got, oracle.sample_tokens(p, u))
    assert list(got[:4]) == [2, 299, 7, 0]
    one = np.array([[1.0]], dtype=np.float32)
    assert run_sample(one, np.array([0.9], np.float32))[0] == 0
