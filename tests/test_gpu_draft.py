"""GPU parity of the draft step: sd_linear (the skinny projection) and
sd_semi_ar_layer (one pass of the semi-autoregressive layer over the draft
cache) against the float64 oracle.

Tolerances.  sd_linear's inputs are exact bf16 values and it accumulates in
fp32, so its error is fp32 rounding of K-term sums (about 2^-24 sqrt(K) of
the terms): max |gpu - ref| / rms(ref) <= 1e-4.  The layer stores four
intermediates in bf16 as the next projection's input, as a bf16 draft does
(the normed rows, q / k / v, the attention output, the SwiGLU activation).
Each rounding adds a relative error of at most 2^-9 per element (rms about
2^-9 / sqrt(3) = 1.1e-3), which the random-like projections carry into the
outputs at about the same relative size; four of them in quadrature give an
rms error near 2.3e-3 of rms(out) and a maximum a few times that over
10^5 - 10^6 elements.  Bounds: rms error <= 5e-3 and max error <= 2.5e-2,
both relative to rms(out).  An appended cache entry is a bf16 value: its
storage rounding is at most 2^-9 of itself, on top of the upstream error of
the projection (rms about 1.1e-3, at most a few times that, of rms): per
element |gpu - ref| <= 2^-9 |ref| + 1e-2 rms.
"""

import numpy as np
import pytest

import oracle
from paper_2505_12728_amd import synth
from tests.gpu_util import normalized_max_error, np_to_device, to_device

pytestmark = pytest.mark.gpu

LIN_TOL = 1e-4
LAYER_MAX, LAYER_RMS = 2.5e-2, 5e-3
CACHE_TOL = 1e-2


def _bf16(x):
    return synth.Tensor(np.asarray(x, np.float32), "bf16")


@pytest.mark.parametrize("R,K,N,bias,res", [(1, 256, 1, False, False), (5, 512, 100, True, False),
                                            (36, 8192, 1000, True, True), (128, 1024, 4096, False, True),
                                            (130, 768, 515, True, True), (7, 28672, 64, False, False),
                                            (16, 256, 65536, True, False),
                                            # seven column-owning waves (512 groups of 112 columns),
                                            # the last group ragged
                                            (36, 512, 57304, True, True)])
def test_linear_parity(R, K, N, bias, res):
    import torch
    import paper_2505_12728_amd as sd
    rng = np.random.default_rng(R * 7 + K + N)
    x = _bf16(rng.normal(size=(R, K)))
    w = _bf16(rng.normal(size=(N, K)) / np.sqrt(K))
    b = rng.normal(size=N).astype(np.float32) if bias else None
    r = rng.normal(size=(R, N)).astype(np.float32) if res else None
    y = sd.sd_linear(to_device(x), to_device(w), None if b is None else np_to_device(b),
                     None if r is None else np_to_device(r))
    torch.cuda.synchronize()
    ref = oracle.linear(x.values, w.values, b, r)
    err, _ = normalized_max_error(y.cpu().numpy(), ref)
    assert err <= LIN_TOL, (R, K, N, err)


def _run_layer(inp, B=None):
    import torch
    import paper_2505_12728_amd as sd
    W = {k: (to_device(v) if isinstance(v, synth.Tensor) else np_to_device(v)) for k, v in inp["weights"].items()}
    kc, vc = to_device(inp["k_cache"]), to_device(inp["v_cache"])
    out = sd.sd_semi_ar_layer(to_device(inp["u"]), W, kc, vc, np_to_device(inp["pos"]), inp["hq"], inp["hkv"],
                              inp["eps"], inp["theta"])
    torch.cuda.synchronize()
    f32 = lambda t: t.float().cpu().numpy()
    return out.cpu().numpy(), f32(kc), f32(vc)


def _check_layer(inp, got):
    out, kc, vc = got
    W = {k: (v.values if isinstance(v, synth.Tensor) else v) for k, v in inp["weights"].items()}
    ref, rk, rv = oracle.semi_ar_layer(inp["u"].values, W, inp["k_cache"].values, inp["v_cache"].values,
                                       inp["pos"], inp["hq"], inp["hkv"], inp["eps"], inp["theta"])
    err, rms = normalized_max_error(out, ref)
    rms_err = float(np.sqrt(np.mean((out - ref) ** 2))) / rms
    assert err <= LAYER_MAX and rms_err <= LAYER_RMS, (err, rms_err)
    r = inp["u"].shape[1]
    for b, p in enumerate(inp["pos"].tolist()):
        # context untouched, new entries close to the oracle's, the rest untouched
        assert np.array_equal(kc[b, :p], inp["k_cache"].values[b, :p])
        assert np.array_equal(vc[b, p + r:], inp["v_cache"].values[b, p + r:])
        for got_c, want in ((kc, rk), (vc, rv)):
            g, ref_c = got_c[b, p:p + r].astype(np.float64), want[b, p:p + r]
            rms_c = float(np.sqrt(np.mean(ref_c ** 2)))
            excess = np.abs(g - ref_c) - (2.0 ** -9 * np.abs(ref_c) + CACHE_TOL * rms_c)
            assert np.all(excess <= 0), (b, float(np.max(excess)) / rms_c)
    return err, rms_err


@pytest.mark.parametrize("name", ["tiny-f32", "llava-7b-image", "qwen2vl-7b-video", "batched-paged"])
def test_semi_ar_layer_workloads(name):
    w = synth.workload(name)
    inp = synth.draft_inputs(w)
    _check_layer(inp, _run_layer(inp))


def test_semi_ar_layer_long_video_shapes():
    # the benchmark's shapes (d = 8192, 64 / 8 heads, I = 28672) on one sequence
    w = synth.workload("long-video")
    inp = synth.draft_inputs(w, batch=1)
    _check_layer(inp, _run_layer(inp))


@pytest.mark.parametrize("B,r,hq,hkv,D,I,ctx", [(3, 1, 4, 4, 64, 256, 0), (2, 16, 2, 1, 128, 512, 5),
                                                (5, 4, 8, 2, 64, 768, 31)])
def test_semi_ar_layer_edge_shapes(B, r, hq, hkv, D, I, ctx):
    # a single new row, an empty context, the largest block (16 rows), MHA
    # and GQA, ragged contexts
    d = hq * D
    w = synth.Workload("edge", "bf16", batch=B, hq=hq, hkv=hkv, head_dim=D, kv_len=64, block=r - 1,
                       draft_ffn=I, draft_ctx=ctx)
    inp = synth.draft_inputs(w, seed=1234 + B + r)
    assert inp["u"].shape == (B, r, 2 * d)
    _check_layer(inp, _run_layer(inp))


def test_semi_ar_layer_deterministic():
    w = synth.workload("qwen2vl-7b-video")
    inp = synth.draft_inputs(w)
    a = _run_layer(inp)
    b = _run_layer(inp)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
