"""GPU parity of the int8 draft (weight-only int8 rows with one fp32 scale
each): sd_linear_q8 and sd_semi_ar_layer_q8 against the oracle on the
dequantised weights.  The int8 x bf16 products are exact in the fp32
accumulation and each output is scaled once, so the bounds are those of the
bf16 path (test_gpu_draft.py): sd_linear_q8 max error <= 1e-4 of rms; the
layer rms error <= 5e-3 and max error <= 2.5e-2 of rms(out)."""

import numpy as np
import pytest

import oracle
from paper_2505_12728_amd import synth
from tests.gpu_util import normalized_max_error, np_to_device, to_device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("R,K,N,bias,res", [(1, 256, 1, False, False), (9, 512, 100, True, False),
                                            (36, 8192, 1000, True, True), (130, 768, 515, False, True),
                                            (16, 256, 65536, True, False), (36, 512, 57304, False, True)])
def test_linear_q8_parity(R, K, N, bias, res):
    import torch
    import paper_2505_12728_amd as sd
    rng = np.random.default_rng(R + 3 * K + N)
    x = synth.Tensor(rng.normal(size=(R, K)).astype(np.float32), "bf16")
    wq = rng.integers(-128, 128, size=(N, K)).astype(np.int8)
    sc = (rng.uniform(0.5, 2.0, size=N) / (80.0 * np.sqrt(K))).astype(np.float32)
    b = rng.normal(size=N).astype(np.float32) if bias else None
    r = rng.normal(size=(R, N)).astype(np.float32) if res else None
    y = sd.sd_linear_q8(to_device(x), np_to_device(wq), np_to_device(sc), None if b is None else np_to_device(b),
                        None if r is None else np_to_device(r))
    torch.cuda.synchronize()
    err, _ = normalized_max_error(y.cpu().numpy(), oracle.linear_q8(x.values, wq, sc, b, r))
    assert err <= 1e-4, (R, K, N, err)


def _run(inp):
    import torch
    import paper_2505_12728_amd as sd
    W = {k: (to_device(v) if isinstance(v, synth.Tensor) else np_to_device(v)) for k, v in inp["weights"].items()}
    kc, vc = to_device(inp["k_cache"]), to_device(inp["v_cache"])
    out = sd.sd_semi_ar_layer_q8(to_device(inp["u"]), W, kc, vc, np_to_device(inp["pos"]), inp["hq"], inp["hkv"],
                                 inp["eps"], inp["theta"])
    torch.cuda.synchronize()
    return out.cpu().numpy(), kc.float().cpu().numpy(), vc.float().cpu().numpy()


@pytest.mark.parametrize("name,batch", [("tiny-f32", None), ("qwen2vl-7b-video", None), ("batched-paged", None),
                                        ("long-video", 1)])
def test_semi_ar_layer_q8_parity(name, batch):
    w = synth.workload(name)
    inp = synth.draft_inputs(w, batch=batch, q8=True)
    out, kc, vc = _run(inp)
    ref, rk, rv = oracle.semi_ar_layer_q8(inp["u"].values, inp["weights"], inp["k_cache"].values,
                                          inp["v_cache"].values, inp["pos"], inp["hq"], inp["hkv"], inp["eps"],
                                          inp["theta"])
    err, rms = normalized_max_error(out, ref)
    rms_err = float(np.sqrt(np.mean((out - ref) ** 2))) / rms
    assert err <= 2.5e-2 and rms_err <= 5e-3, (err, rms_err)
    r = inp["u"].shape[1]
    for b, p in enumerate(inp["pos"].tolist()):
        for got, want in ((kc, rk), (vc, rv)):
            g, rc = got[b, p:p + r].astype(np.float64), want[b, p:p + r]
            rms_c = float(np.sqrt(np.mean(rc ** 2)))
            assert np.all(np.abs(g - rc) <= 2.0 ** -9 * np.abs(rc) + 1e-2 * rms_c)


def test_q8_and_bf16_layers_agree_on_the_same_weights():
    # the bf16 draft holding the dequantised weights (exact in bf16 when the
    # scales are powers of two) gives the same outputs as the int8 draft
    import torch
    import paper_2505_12728_amd as sd
    w = synth.workload("tiny-f32")
    inp = synth.draft_inputs(w, q8=True)
    for name in oracle.draft_layer.Q8_WEIGHTS:
        inp["weights"][name + "_s"] = np.full_like(inp["weights"][name + "_s"], 2.0 ** -10)
    out_q, _, _ = _run(inp)
    Wb = {k: v for k, v in inp["weights"].items() if not k.endswith("_s")}
    for name in oracle.draft_layer.Q8_WEIGHTS:
        Wb[name] = synth.Tensor((inp["weights"][name].astype(np.float32) * 2.0 ** -10), "bf16")
    Wd = {k: (to_device(v) if isinstance(v, synth.Tensor) else np_to_device(v)) for k, v in Wb.items()}
    out_b = sd.sd_semi_ar_layer(to_device(inp["u"]), Wd, to_device(inp["k_cache"]), to_device(inp["v_cache"]),
                                np_to_device(inp["pos"]), inp["hq"], inp["hkv"], inp["eps"], inp["theta"])
    torch.cuda.synchronize()
    assert np.array_equal(out_q, out_b.cpu().numpy())
