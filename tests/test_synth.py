"""Checks of the seeded input generator (CPU only)."""

import math

import numpy as np
import torch

from paper_2505_12728_amd import synth


def test_bf16_rounding_matches_torch():
    r = np.random.default_rng(0)
    x = np.concatenate([r.standard_normal(100000).astype(np.float32) * 10,
                        np.array([1.0, -2.5, 3.140625, 65504.0, 1e-30, 0.0], np.float32)])
    ours = synth.bf16_bits(x)
    theirs = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, theirs)
    np.testing.assert_array_equal(synth.bf16_to_f32(ours),
                                  torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_inputs_are_deterministic_and_shaped():
    w = synth.workload(0)
    a = synth.verify_inputs(w)
    b = synth.verify_inputs(w)
    np.testing.assert_array_equal(a["q"].values, b["q"].values)
    assert a["q"].shape == (1, 4, 4, 64)
    assert a["k_cache"].shape == (1, 608, 1, 64)
    lat, feats = synth.compress_inputs(w)
    assert lat.shape == (16, 256) and feats.shape == (1, 576, 256)
    acc = synth.accept_inputs(w, "sampled")
    assert acc["p"].shape == (1, 5, 1024) and acc["q"].shape == (1, 4, 1024)
    np.testing.assert_allclose(acc["p"].sum(-1), 1.0, atol=1e-5)
    u = acc["u"].astype(np.float64) * 2 ** 24
    assert np.all(u == np.floor(u)) and np.all(u < 2 ** 24)


def test_paged_layout_covers_each_token_once():
    w = synth.Workload("paged-small", "bf16", batch=3, hq=4, hkv=2, head_dim=8,
                       kv_len=100, kv_len_min=20, block=3, paged=True)
    d = synth.verify_inputs(w, seed=5)
    lens = d["kv_len"]
    table = d["page_table"]
    owned = set()
    for b, L in enumerate(lens):
        for i in range(math.ceil(int(L) / 16)):
            assert int(table[b, i]) not in owned
            owned.add(int(table[b, i]))
    pool = d["k_cache"].values
    spare = [p for p in range(pool.shape[0]) if p not in owned]
    assert np.all(pool[spare] == synth.POISON)
