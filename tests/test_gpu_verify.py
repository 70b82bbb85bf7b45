"""GPU parity of sd_verify_attention against the oracle (same seeded inputs)."""

import math

import numpy as np
import pytest

import oracle
from paper_2505_12728_amd import synth
from tests.gpu_util import assert_close, assert_lse_close, np_to_device, to_device

pytestmark = pytest.mark.gpu


def run_gpu(d, scale=None):
    import torch
    import paper_2505_12728_amd as sd
    q = to_device(d["q"])
    kc = to_device(d["k_cache"])
    vc = to_device(d["v_cache"])
    kl = np_to_device(d["kv_len"].astype(np.int32))
    pt = None if d["page_table"] is None else np_to_device(d["page_table"].astype(np.int32))
    out, lse = sd.sd_verify_attention(q, kc, vc, kl, scale=scale, page_table=pt)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


def oracle_slice(d, b, hk, g, scale):
    """Oracle for one (sequence, KV head): its g query heads over its cache."""
    q = d["q"].values[b:b + 1, :, hk * g:(hk + 1) * g]
    if d["page_table"] is None:
        kc = d["k_cache"].values[b:b + 1, :, hk:hk + 1]
        vc = d["v_cache"].values[b:b + 1, :, hk:hk + 1]
        return oracle.verify_attention(q, kc, vc, d["kv_len"][b:b + 1], scale)
    kc = d["k_cache"].values[:, hk:hk + 1]
    vc = d["v_cache"].values[:, hk:hk + 1]
    return oracle.verify_attention(q, kc, vc, d["kv_len"][b:b + 1], scale,
                                   page_table=d["page_table"][b:b + 1])


def check_pairs(d, w, out, lse, pairs, dtype):
    scale = 1.0 / math.sqrt(w.head_dim)
    g = w.hq // w.hkv
    for b, hk in pairs:
        ro, rl = oracle_slice(d, b, hk, g, scale)
        assert_close(out[b:b + 1, :, hk * g:(hk + 1) * g], ro, dtype, f"out b={b} hk={hk}")
        assert_lse_close(lse[b:b + 1, :, hk * g:(hk + 1) * g], rl, dtype, f"lse b={b} hk={hk}")


@pytest.mark.parametrize("wi", [0, 1, 2])
def test_verify_workload_full_oracle(wi):
    w = synth.workload(wi)
    print(f"verify workload {w.name}", flush=True)
    d = synth.verify_inputs(w)
    out, lse = run_gpu(d)
    ro, rl = oracle.verify_attention(d["q"].values, d["k_cache"].values, d["v_cache"].values,
                                     d["kv_len"], 1.0 / math.sqrt(w.head_dim))
    assert_close(out, ro, w.dtype, w.name)
    assert_lse_close(lse, rl, w.dtype, w.name)


def oracle_full(d, w, scale):
    """Oracle outputs of a whole workload, assembled from one oracle call per
    sequence (paged) or per (sequence, KV head) (contiguous), so that every
    element of the device's output is compared."""
    B, k, Hq, D = d["q"].shape
    g = w.hq // w.hkv
    out = np.zeros((B, k, Hq, D))
    lse = np.zeros((B, k, Hq))
    if d["page_table"] is not None:
        kp = np.asarray(d["k_cache"].values, np.float64)
        vp = np.asarray(d["v_cache"].values, np.float64)
        for b in range(B):
            o, l = oracle.verify_attention(d["q"].values[b:b + 1], kp, vp, d["kv_len"][b:b + 1],
                                           scale, page_table=d["page_table"][b:b + 1])
            out[b], lse[b] = o[0], l[0]
        return out, lse
    for b in range(B):
        for hk in range(w.hkv):
            hs = slice(hk * g, (hk + 1) * g)
            o, l = oracle_slice(d, b, hk, g, scale)
            out[b, :, hs], lse[b, :, hs] = o[0], l[0]
    return out, lse


@pytest.mark.parametrize("wi", [3, 4])
def test_verify_long_kv_workload_every_element(wi):
    # batched-paged (16 ragged paged sequences) and long-video (4 x 65536) at
    # full size, in the launch configuration the benchmark times; every
    # (sequence, KV head) pair is compared, so work-groups whose key range
    # spans several pairs and the XCD-ordered grid are all covered
    w = synth.workload(wi)
    print(f"verify workload {w.name}", flush=True)
    d = synth.verify_inputs(w)
    out, lse = run_gpu(d)
    ro, rl = oracle_full(d, w, 1.0 / math.sqrt(w.head_dim))
    assert_close(out, ro, w.dtype, w.name)
    assert_lse_close(lse, rl, w.dtype, w.name)
    # the per-pair bound holds too (no pair hides behind the whole-tensor rms)
    check_pairs(d, w, out, lse, [(0, 0), (w.batch - 1, w.hkv - 1)], w.dtype)


CASES = [
    # name, dtype, B, k, Hq, Hkv, D, lens, paged
    ("ragged-tail", "bf16", 2, 3, 8, 2, 128, [1000, 517], False),
    ("single-key", "bf16", 1, 1, 4, 4, 128, [1], False),
    ("short-rows-empty", "bf16", 2, 5, 4, 1, 128, [3, 0], False),
    ("head-dim-64", "bf16", 2, 4, 12, 3, 64, [700, 130], False),
    ("mha-one-row", "bf16", 1, 1, 8, 8, 128, [4096], False),
    ("two-row-groups", "bf16", 1, 16, 8, 1, 128, [777], False),
    ("paged-ragged", "bf16", 3, 6, 8, 2, 128, [33, 1000, 2049], True),
    ("paged-d64", "bf16", 2, 2, 4, 2, 64, [17, 300], True),
    # 3-4 row blocks per KV head: 8 waves in two key groups
    ("rows64-ragged", "bf16", 2, 8, 16, 2, 128, [1000, 37], False),
    ("rows48-short", "bf16", 1, 6, 8, 1, 128, [70], False),
    ("rows64-d64", "bf16", 2, 8, 8, 1, 64, [2500, 64], False),
    ("rows64-paged", "bf16", 2, 8, 16, 2, 128, [300, 1500], True),
    # a few tiles per work-group: two key groups whose ranges span pairs
    # (one group of a one-tile range gets no tile), and paged ragged rows
    ("multi-pair-rows64-kg2", "bf16", 3, 8, 16, 2, 128, [1024, 200, 1], False),
    ("multi-pair-paged-rows32", "bf16", 4, 6, 16, 4, 128, [1000, 16, 512, 999], True),
    # 47 key splits: an odd count above 32 in one 64-split chunk of the merge
    ("merge-odd-47", "bf16", 1, 4, 4, 1, 128, [1500], False),
    ("f32-ragged", "f32", 2, 4, 8, 2, 64, [608, 99], False),
    ("f32-paged", "f32", 2, 3, 4, 1, 128, [50, 700], True),
    ("f32-empty-rows", "f32", 1, 4, 4, 1, 64, [2], False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_verify_edge_cases(case):
    name, dt, B, k, Hq, Hkv, D, lens, paged = case
    print(f"verify case {name}", flush=True)
    w = synth.Workload(name, dt, batch=B, hq=Hq, hkv=Hkv, head_dim=D,
                       kv_len=max(max(lens), 1), block=k, paged=paged)
    d = synth.verify_inputs(w, seed=11, kv_len=np.array(lens, np.int32))
    scale = 0.7 / math.sqrt(D)
    out, lse = run_gpu(d, scale=scale)
    if paged:
        ro, rl = oracle.verify_attention(d["q"].values, d["k_cache"].values, d["v_cache"].values,
                                         d["kv_len"], scale, page_table=d["page_table"])
    else:
        ro, rl = oracle.verify_attention(d["q"].values, d["k_cache"].values, d["v_cache"].values,
                                         d["kv_len"], scale)
    if np.any(ro != 0):
        assert_close(out, ro, dt, name)
    else:
        assert np.all(out == 0)
    assert_lse_close(lse, rl, dt, name)
    # rows without a visible key are exactly zero
    assert np.all(out[np.isneginf(rl)] == 0)


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("mult", [-0.9, 0.0, 4.0])
def test_verify_scale_sign_and_size(mult, dt, paged):
    # a negative scale (folded into the queries), a zero scale (every
    # visible key weighs the same) and a large one (the running maximum is
    # raised on many tiles), on ragged lengths with a causal tail
    D = 128
    name = f"scale{mult}-{dt}-{'paged' if paged else 'contiguous'}"
    print(f"verify case {name}", flush=True)
    lens = [700, 33, 1]
    w = synth.Workload(name, dt, batch=3, hq=8, hkv=2, head_dim=D, kv_len=max(lens), block=5,
                       paged=paged)
    d = synth.verify_inputs(w, seed=23, kv_len=np.array(lens, np.int32))
    scale = mult / math.sqrt(D)
    out, lse = run_gpu(d, scale=scale)
    kw = {"page_table": d["page_table"]} if paged else {}
    ro, rl = oracle.verify_attention(d["q"].values, d["k_cache"].values, d["v_cache"].values,
                                     d["kv_len"], scale, **kw)
    assert_close(out, ro, dt, name)
    assert_lse_close(lse, rl, dt, name)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_verify_beyond_grid_extent(dt):
    # 70000 (sequence, KV head) pairs: more than a grid's y extent (65535)
    # holds, on every kernel of the path (merges included)
    B = 70000
    print(f"verify grid case {dt} B={B}", flush=True)
    lens = np.random.default_rng(41).integers(0, 40, size=B).astype(np.int32)
    w = synth.Workload("many-pairs", dt, batch=B, hq=2, hkv=1, head_dim=64, kv_len=40, block=1)
    d = synth.verify_inputs(w, seed=43, kv_len=lens)
    scale = 1 / 8
    out, lse = run_gpu(d, scale=scale)
    ro, rl = oracle.verify_attention(d["q"].values, d["k_cache"].values, d["v_cache"].values,
                                     d["kv_len"], scale)
    assert_close(out, ro, dt, "many-pairs")
    assert_lse_close(lse, rl, dt, "many-pairs")
    assert np.all(out[lens == 0] == 0)


@pytest.mark.parametrize("paged", [False, True])
def test_verify_workspace_reuse_short_and_empty_sequences(paged):
    # a 16K-capacity cache holding short sequences (fewer tiles than
    # work-groups, so some work-groups have no range), empty sequences
    # between non-empty ones, and one workspace reused over calls of
    # different lengths
    import torch
    import paper_2505_12728_amd as sd
    print(f"verify reuse paged={paged}", flush=True)
    scale = 1 / math.sqrt(128)
    cases = [[40, 0, 3, 0, 65], [0, 0, 1, 0, 0], [700, 0, 16384, 31, 0], [40, 0, 3, 0, 65]]
    w = synth.Workload("reuse", "bf16", batch=5, hq=8, hkv=2, head_dim=128, kv_len=16384, block=3,
                       paged=paged)
    ws = None
    for i, lens in enumerate(cases):
        d = synth.verify_inputs(w, seed=50 + i, kv_len=np.array(lens, np.int32))
        q, kc, vc = to_device(d["q"]), to_device(d["k_cache"]), to_device(d["v_cache"])
        kl = np_to_device(d["kv_len"].astype(np.int32))
        pt = None if d["page_table"] is None else np_to_device(d["page_table"].astype(np.int32))
        if ws is None:
            cap = 16384
            n = sd.sd_verify_workspace_size(5, 3, 8, 2, 128, cap, sd.SD_BF16)
            ws = torch.zeros(n, dtype=torch.uint8, device="cuda")
        out, lse = sd.sd_verify_attention(q, kc, vc, kl, scale=scale, page_table=pt, workspace=ws)
        torch.cuda.synchronize()
        kw = {} if d["page_table"] is None else {"page_table": d["page_table"]}
        ro, rl = oracle.verify_attention(d["q"].values, d["k_cache"].values, d["v_cache"].values,
                                         d["kv_len"], scale, **kw)
        out, lse = out.cpu().numpy(), lse.cpu().numpy()
        empty = np.array(lens) == 0
        assert np.all(out[empty] == 0) and np.all(np.isneginf(lse[empty])), f"call {i}"
        if np.any(ro != 0):
            assert_close(out, ro, "bf16", f"reuse call {i}")
        assert_lse_close(lse, rl, "bf16", f"reuse call {i}")


def test_verify_nan_poison_beyond_length_is_never_read():
    w = synth.Workload("poison", "bf16", batch=2, hq=8, hkv=2, head_dim=128, kv_len=640, block=4)
    lens = np.array([600, 333], np.int32)
    clean = synth.verify_inputs(w, seed=3, kv_len=lens)
    dirty = synth.verify_inputs(w, seed=3, kv_len=lens, poison=float("nan"))
    a, la = run_gpu(clean)
    b, lb = run_gpu(dirty)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_verify_paged_equals_contiguous_bitwise():
    import torch
    import paper_2505_12728_amd as sd
    rng = np.random.default_rng(5)
    B, k, Hq, Hkv, D = 3, 5, 16, 4, 128
    lens = np.array([1111, 40, 2000], np.int32)
    Lmax = 2048
    kf = synth.Tensor(rng.standard_normal((B, Lmax, Hkv, D)).astype(np.float32), "bf16")
    vf = synth.Tensor(rng.standard_normal((B, Lmax, Hkv, D)).astype(np.float32), "bf16")
    q = synth.Tensor(rng.standard_normal((B, k, Hq, D)).astype(np.float32), "bf16")
    pages = (lens + 15) // 16
    n_pool = int(pages.sum()) + 5
    perm = rng.permutation(n_pool)
    table = np.zeros((B, Lmax // 16), np.int32)
    kb = np.zeros((n_pool, Hkv, 16, D), np.uint16)
    vb = np.zeros((n_pool, Hkv, 16, D), np.uint16)
    pos = 0
    for b in range(B):
        for i in range(pages[b]):
            pg = perm[pos]
            pos += 1
            table[b, i] = pg
            kb[pg] = kf.bits[b, i * 16:(i + 1) * 16].transpose(1, 0, 2)
            vb[pg] = vf.bits[b, i * 16:(i + 1) * 16].transpose(1, 0, 2)
    to_bf = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    kl = np_to_device(lens)
    o1, l1 = sd.sd_verify_attention(to_device(q), to_device(kf), to_device(vf), kl)
    o2, l2 = sd.sd_verify_attention(to_device(q), to_bf(kb), to_bf(vb), kl,
                                    page_table=np_to_device(table))
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_verify_is_deterministic():
    w = synth.workload(2)
    d = synth.verify_inputs(w)
    a, la = run_gpu(d)
    b, lb = run_gpu(d)
    assert np.array_equal(a, b) and np.array_equal(la, lb)



def test_verify_f32_unaligned_bases():
    # fp32 caches and queries need only 4-byte alignment: bases 4 bytes off
    # a 16-byte boundary take the kernel's 4-byte staging loads
    import torch
    import paper_2505_12728_amd as sd
    print("verify f32 unaligned bases", flush=True)
    lens = [300, 77]
    w = synth.Workload("f32-unaligned", "f32", batch=2, hq=8, hkv=2, head_dim=64, kv_len=300, block=3)
    d = synth.verify_inputs(w, seed=91, kv_len=np.array(lens, np.int32))

    def shifted(x):
        x = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
        buf = torch.empty(x.numel() + 1, dtype=torch.float32, device="cuda")
        t = buf[1:].view(x.shape)
        t.copy_(x.cuda())
        assert t.data_ptr() % 16 == 4
        return t
    q, kc, vc = shifted(d["q"].values), shifted(d["k_cache"].values), shifted(d["v_cache"].values)
    kl = np_to_device(d["kv_len"].astype(np.int32))
    scale = 1 / 8
    out, lse = sd.sd_verify_attention(q, kc, vc, kl, scale=scale)
    torch.cuda.synchronize()
    ro, rl = oracle.verify_attention(d["q"].values, d["k_cache"].values, d["v_cache"].values, d["kv_len"], scale)
    assert_close(out.cpu().numpy(), ro, "f32", "f32-unaligned")
    assert_lse_close(lse.cpu().numpy(), rl, "f32", "f32-unaligned")
