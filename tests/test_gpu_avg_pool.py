"""GPU parity of sd_avg_pool_compress against the oracle: sums in float64
and one rounding to float32, so max |gpu - ref| / rms(ref) <= 1e-6."""

import numpy as np
import pytest

import oracle
from paper_2505_12728_amd import synth
from tests.gpu_util import normalized_max_error, to_device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("B,N,C,d,dtype", [(1, 576, 64, 4096, "bf16"), (2, 7, 3, 5, "f32"), (3, 1000, 1, 256, "bf16"),
                                           (1, 100, 100, 24, "bf16"), (4, 16384, 512, 8192, "bf16"),
                                           (2, 33, 8, 1030, "f32")])
def test_avg_pool_parity(B, N, C, d, dtype):
    import torch
    import paper_2505_12728_amd as sd
    rng = np.random.default_rng(B * N + C + d)
    F = synth.Tensor(rng.normal(size=(B, N, d)).astype(np.float32), dtype)
    out = sd.sd_avg_pool_compress(to_device(F), C)
    torch.cuda.synchronize()
    err, _ = normalized_max_error(out.cpu().numpy(), oracle.avg_pool_compress(F.values, C))
    assert err <= 1e-6, err
