"""sd_spec_accept_noalloc (the acceptance rule with the library's fixed
device scratch, for callers that cannot allocate) against sd_spec_accept:
identical results, called through the C ABI, on two calls in a row with the
second smaller, in both modes."""

import ctypes

import numpy as np
import pytest

from paper_2505_12728_amd import synth
from tests.gpu_util import np_to_device

pytestmark = pytest.mark.gpu


def noalloc(p, q, draft, u, mode):
    import torch
    import paper_2505_12728_amd as sd
    B, kp1, V = p.shape
    n = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    t = torch.full((B, kp1), -7, dtype=torch.int32, device="cuda")
    ptr = lambda x: None if x is None else ctypes.c_void_p(x.data_ptr())
    st = sd.library().sd_spec_accept_noalloc(ptr(p), ptr(q), ptr(draft), ptr(u), ptr(n), ptr(t), B,
                                             kp1 - 1, V, mode,
                                             ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == sd.SD_OK, sd.sd_status_string(st)
    return n, t


def with_workspace(p, q, draft, u, mode):
    import paper_2505_12728_amd as sd
    return sd.sd_spec_accept(p, q, draft, u, mode)


def inputs(wi, mode, batch, seed):
    w = synth.workload(wi)
    a = synth.accept_inputs(w, "sampled" if mode == 1 else "greedy", seed=seed, batch=batch)
    q = np_to_device(a["q"]) if mode == 1 else None
    u = np_to_device(a["u"]) if mode == 1 else None
    return np_to_device(a["p"]), q, np_to_device(a["draft"]), u


@pytest.mark.parametrize("mode", [1, 0])
def test_noalloc_matches_workspace_entry_point(mode):
    import torch
    # a large call (16 sequences over a 152064-token vocabulary), then a
    # smaller one (3 sequences, 32000 tokens, other k) on the same scratch
    for wi, batch, seed in [(2, 16, 5), (1, 3, 6), (4, 4, 7)]:
        p, q, draft, u = inputs(wi, mode, batch, seed)
        print(f"noalloc mode {mode} workload {wi} batch {batch}", flush=True)
        n1, t1 = noalloc(p, q, draft, u, mode)
        n2, t2 = with_workspace(p, q, draft, u, mode)
        torch.cuda.synchronize()
        assert torch.equal(n1, n2) and torch.equal(t1, t2), (wi, batch)
        assert int(n1.min()) >= 0


def test_noalloc_repeated_calls_on_one_stream():
    import torch
    p, q, draft, u = inputs(3, 1, 16, 9)
    ref = with_workspace(p, q, draft, u, 1)
    for _ in range(5):
        n, t = noalloc(p, q, draft, u, 1)
    torch.cuda.synchronize()
    assert torch.equal(n, ref[0]) and torch.equal(t, ref[1])
