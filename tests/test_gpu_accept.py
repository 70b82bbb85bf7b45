"""GPU parity of sd_spec_accept: bit-exact against the oracle."""

import json
import os

import numpy as np
import pytest

import oracle
from paper_2505_12728_amd import synth
from tests.gpu_util import np_to_device

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def run_gpu(p, q, draft, u, mode):
    import torch
    import paper_2505_12728_amd as sd
    B, kp1, V = p.shape
    qd = np_to_device(q.astype(np.float32)) if q is not None else None
    ud = np_to_device(u.astype(np.float32)) if u is not None else None
    n, t = sd.sd_spec_accept(np_to_device(p.astype(np.float32)), qd,
                             np_to_device(draft.astype(np.int32)), ud, mode)
    torch.cuda.synchronize()
    return n.cpu().numpy(), t.cpu().numpy()


def check(p, q, draft, u, mode, what):
    n, t = run_gpu(p, q, draft, u, mode)
    rn, rt = oracle.spec_accept(p, q, draft, u, mode)
    assert np.array_equal(n, rn), f"{what}: n {n} vs oracle {rn}"
    assert np.array_equal(t, rt), f"{what}: tokens differ\n{t}\n{rt}"
    return n


@pytest.mark.parametrize("wi,mode", [(0, "sampled"), (0, "greedy"), (1, "sampled"),
                                     (2, "greedy"), (2, "sampled"), (3, "sampled"),
                                     (4, "sampled")])
def test_accept_workloads_bit_exact(wi, mode):
    w = synth.workload(wi)
    print(f"accept workload {w.name} {mode}", flush=True)
    d = synth.accept_inputs(w, mode)
    m = oracle.ACCEPT_GREEDY if mode == "greedy" else oracle.ACCEPT_SAMPLED
    check(d["p"], d["q"], d["draft"], d["u"], m, f"{w.name}/{mode}")


def test_accept_hand_cases_on_gpu():
    with open(os.path.join(GOLDEN, "accept_hand_cases.json")) as fh:
        cases = json.load(fh)["cases"]
    for c in cases:
        greedy = c["mode"] == "greedy"
        p = np.array(c["p"], np.float32)[None]
        k = p.shape[1] - 1
        q = None if c["q"] is None else np.array(c["q"], np.float32)[None]
        u = None if c["u"] is None else np.array(c["u"], np.float32)[None]
        n, t = run_gpu(p, q, np.array(c["draft"], np.int32)[None], u,
                       oracle.ACCEPT_GREEDY if greedy else oracle.ACCEPT_SAMPLED)
        assert n[0] == c["n"] and list(t[0]) == c["tokens"], c["name"]


def _probs(rng, shape, temp=1.0):
    z = rng.standard_normal(shape) * 3 / temp
    e = np.exp(z - z.max(-1, keepdims=True))
    return (e / e.sum(-1, keepdims=True)).astype(np.float32)


def test_accept_random_batches_both_modes():
    rng = np.random.default_rng(9)
    for (B, k, V) in [(64, 7, 5000), (7, 16, 1 << 18), (33, 1, 3), (5, 3, 1)]:
        p = _probs(rng, (B, k + 1, V))
        q = _probs(rng, (B, k, V))
        draft = rng.integers(0, V, size=(B, k)).astype(np.int32)
        # make some drafts likely to be accepted: copy the target argmax
        draft[:, ::2] = np.argmax(p[:, :k:2], axis=-1)
        u = (rng.integers(0, 1 << 24, size=(B, k + 1)) * 2.0 ** -24).astype(np.float32)
        check(p, q, draft, u, oracle.ACCEPT_SAMPLED, f"sampled B={B} k={k} V={V}")
        check(p, q, draft, u, oracle.ACCEPT_GREEDY, f"greedy B={B} k={k} V={V}")


def test_accept_beyond_grid_extent():
    # 66000 sequences: more than a grid's y extent (65535)
    rng = np.random.default_rng(47)
    B, k, V = 66000, 1, 5
    print(f"accept grid case B={B}", flush=True)
    p = _probs(rng, (B, k + 1, V))
    q = _probs(rng, (B, k, V))
    draft = rng.integers(0, V, size=(B, k)).astype(np.int32)
    u = (rng.integers(0, 1 << 24, size=(B, k + 1)) * 2.0 ** -24).astype(np.float32)
    check(p, q, draft, u, oracle.ACCEPT_SAMPLED, f"sampled B={B}")
    check(p, q, draft, u, oracle.ACCEPT_GREEDY, f"greedy B={B}")


def test_accept_draft_equal_to_target_accepts_all():
    rng = np.random.default_rng(10)
    B, k, V = 16, 6, 32000
    p = _probs(rng, (B, k + 1, V))
    draft = np.argmax(p[:, :k], axis=-1).astype(np.int32)
    u = (rng.integers(0, 1 << 24, size=(B, k + 1)) * 2.0 ** -24).astype(np.float32)
    n = check(p, p[:, :k].copy(), draft, u, oracle.ACCEPT_SAMPLED, "q=p")
    assert np.all(n == k)


def test_accept_planted_greedy_mismatches():
    rng = np.random.default_rng(12)
    B, k, V = 9, 8, 4096
    p = _probs(rng, (B, k + 1, V))
    g = np.argmax(p, axis=-1)
    draft = g[:, :k].astype(np.int32).copy()
    for b in range(B):
        if b < k:
            draft[b, b] = (draft[b, b] + 1) % V
    n = check(p, None, draft, None, oracle.ACCEPT_GREEDY, "planted")
    assert list(n) == list(range(k)) + [k]


def test_accept_invalid_ids_and_degenerate_rows():
    rng = np.random.default_rng(13)
    B, k, V = 6, 4, 777
    p = _probs(rng, (B, k + 1, V))
    q = _probs(rng, (B, k, V))
    draft = rng.integers(0, V, size=(B, k)).astype(np.int32)
    draft[0, 0] = -5
    draft[1, 2] = V + 3
    # sequence 2: unnormalised rejected row with no residual mass
    p[2, 0] = 0.0
    p[2, 0, 10] = 1e-3
    q[2, 0] = 0.5
    # sequence 3: all-zero target row at the rejection point -> argmax fallback
    p[3, 0] = 0.0
    q[3, 0] = 0.25
    u = (rng.integers(0, 1 << 24, size=(B, k + 1)) * 2.0 ** -24).astype(np.float32)
    u[2, 0] = 0.999
    u[3, 0] = 0.999
    check(p, q, draft, u, oracle.ACCEPT_SAMPLED, "degenerate")
    check(p, q, draft, u, oracle.ACCEPT_GREEDY, "degenerate-greedy")
