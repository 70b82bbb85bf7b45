"""Shared helpers of the GPU parity tests (inputs to the device, error norms)."""

import numpy as np

# Float tolerance: max |gpu - oracle| / rms(oracle) per output tensor, i.e.
# the max-abs error after scaling the reference output to unit variance:
# 5e-3 for bf16 inputs (fp32 accumulation), 1e-5 for fp32 inputs.
TOL = {"bf16": 5e-3, "f32": 1e-5}
# lse is a log-domain scalar of size O(log L + |s|); absolute bound
LSE_TOL = {"bf16": 1e-3, "f32": 1e-5}
# Probability vectors (the LM head's softmax): per entry
# |p_gpu - p_ref| <= rel * p_ref + abs.  The inputs are exact in float32, so
# the error is the float32 accumulation of the d-term logit (about
# 2^-24 sqrt(d) times the size of the terms: ~2e-5 at d = 8192) divided by
# tau, plus a few ulp in the exponent; rel = 2e-3 bounds the logit error to
# 2e-3 tau with a wide margin.  fp32 inputs are summed in float64.  (A
# max / rms norm grows like sqrt(V) for peaked distributions, so it is not
# used for them.)
PROB_TOL = {"bf16": (2e-3, 1e-7), "f32": (1e-5, 1e-12)}


def to_device(t):
    """synth.Tensor -> torch tensor on cuda:0 holding exactly the same values."""
    import torch
    if t.dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(t.bits).view(np.int16)).view(
            torch.bfloat16).to("cuda")
    return torch.from_numpy(np.ascontiguousarray(t.values)).to("cuda")


def np_to_device(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def normalized_max_error(gpu, ref):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    return float(np.max(np.abs(gpu - ref))) / max(rms, 1e-30), rms


def assert_close(gpu, ref, dtype, what):
    err, rms = normalized_max_error(gpu, ref)
    raw = float(np.max(np.abs(np.asarray(gpu, np.float64) - np.asarray(ref, np.float64))))
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    assert err <= TOL[dtype], f"{what}: normalised max error {err:.3g} > {TOL[dtype]} " \
                              f"(raw {raw:.3g}, rms {rms:.3g})"
    return err


def assert_lse_close(gpu, ref, dtype, what):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(gpu)), f"{what}: -inf pattern differs"
    if fin.any():
        err = float(np.max(np.abs(gpu[fin] - ref[fin])))
        assert err <= LSE_TOL[dtype], f"{what}: lse error {err:.3g}"


def assert_probs_close(gpu, ref, dtype, what):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    rel, ab = PROB_TOL[dtype]
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    excess = np.abs(gpu - ref) - (rel * ref + ab)
    i = np.unravel_index(np.argmax(excess), excess.shape)
    assert excess[i] <= 0, (f"{what}: |gpu - ref| = {abs(gpu[i] - ref[i]):.3g} at {i} "
                            f"(ref {ref[i]:.3g}) exceeds {rel} * ref + {ab}")
    return float(np.max(np.abs(gpu - ref) / (ref + ab)))
