"""The Python binding rejects caller-supplied outputs of the wrong shape,
dtype or device before any C call (a short buffer would otherwise be written
past its end by the kernels)."""

import pytest

pytestmark = pytest.mark.gpu


def _t(shape, dtype="float32", device="cuda"):
    import torch
    return torch.zeros(shape, dtype=getattr(torch, dtype), device=device)


def test_compress_rejects_bad_out():
    import paper_2505_12728_amd as sd
    lat, feats = _t((32, 128), "bfloat16"), _t((2, 64, 128), "bfloat16")
    with pytest.raises(ValueError, match="shape"):
        sd.sd_latent_compress(lat, feats, 1, 1.0, out=_t((2, 31, 128)))
    with pytest.raises(TypeError):
        sd.sd_latent_compress(lat, feats, 1, 1.0, out=_t((2, 32, 128), "bfloat16"))
    with pytest.raises(ValueError, match="GPU"):
        sd.sd_latent_compress(lat, feats, 1, 1.0, out=_t((2, 32, 128), device="cpu"))


def test_verify_rejects_bad_out_and_lse():
    import paper_2505_12728_amd as sd
    q = _t((1, 4, 8, 128), "bfloat16")
    kc = _t((1, 64, 2, 128), "bfloat16")
    kl = _t((1,), "int32")
    kl.fill_(64)
    with pytest.raises(ValueError, match="shape"):
        sd.sd_verify_attention(q, kc, kc, kl, out=_t((1, 4, 8, 64)))
    with pytest.raises(ValueError, match="shape"):
        sd.sd_verify_attention(q, kc, kc, kl, lse=_t((1, 4, 7)))
    with pytest.raises(TypeError):
        sd.sd_verify_attention(q, kc, kc, kl, lse=_t((1, 4, 8), "float64"))


def test_accept_rejects_bad_outputs():
    import paper_2505_12728_amd as sd
    B, k, V = 2, 3, 50
    p, q = _t((B, k + 1, V)), _t((B, k, V))
    draft, u = _t((B, k), "int32"), _t((B, k + 1))
    with pytest.raises(TypeError):
        sd.sd_spec_accept(p, q, draft, u, n_accepted=_t((B,), "int64"))
    with pytest.raises(TypeError):
        sd.sd_spec_accept(p, q, draft, u, tokens=_t((B, k + 1), "int64"))
    with pytest.raises(ValueError, match="shape"):
        sd.sd_spec_accept(p, q, draft, u, tokens=_t((B, k), "int32"))
    with pytest.raises(ValueError, match="shape"):
        sd.sd_spec_accept_logits(p, q, draft, 1, 0, 1.0, n_accepted=_t((1,), "int32"))
    with pytest.raises(ValueError, match="shape"):
        sd.sd_philox_uniforms(1, 0, 2, 5, out=_t((2, 4)))


def test_head_sampling_and_draft_reject_bad_outputs():
    import paper_2505_12728_amd as sd
    h, w = _t((3, 256), "bfloat16"), _t((40, 256), "bfloat16")
    with pytest.raises(ValueError, match="shape"):
        sd.sd_lm_head_probs(h, w, 1.0, out=_t((3, 39)))
    with pytest.raises(ValueError, match="shape"):
        sd.sd_sample_tokens(_t((3, 40)), _t((3,)), out=_t((2,), "int32"))
    x, wl = _t((4, 256), "bfloat16"), _t((64, 256), "bfloat16")
    with pytest.raises(ValueError, match="shape"):
        sd.sd_linear(x, wl, out=_t((4, 63)))
    with pytest.raises(ValueError, match="shape"):
        sd.sd_linear_q8(x, _t((64, 256), "int8"), _t((64,)), out=_t((3, 64)))
    with pytest.raises(ValueError, match="shape"):
        sd.sd_avg_pool_compress(_t((1, 10, 64)), 5, out=_t((1, 4, 64)))
