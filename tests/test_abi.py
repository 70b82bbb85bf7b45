"""C ABI checks that need no GPU: the library loads, exports every symbol
the header declares, and rejects bad arguments before touching HIP."""

import ctypes
import os
import re

import pytest

import paper_2505_12728_amd as sd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specflash.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sd_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(sd.library_path):
        pytest.fail("libspecflash.so is not built (run __graft_entry__.build())")
    return sd.library()


def test_header_declares_the_three_entry_points():
    names = header_functions()
    for n in ["sd_latent_compress", "sd_verify_attention", "sd_spec_accept"]:
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in header_functions():
        assert hasattr(lib, name), name
    assert set(header_functions()) <= set(sd._SIGNATURES)


def test_status_strings_and_version(lib):
    assert sd.sd_status_string(sd.SD_OK) == "SD_OK"
    for s in range(1, 5):
        assert sd.sd_status_string(s).startswith("SD_ERR")
    assert "unknown" in sd.sd_status_string(99)
    assert sd.sd_version() >> 16 == 1


def _fake(n=1):
    # aligned non-null host addresses: validation never dereferences them
    buf = ctypes.create_string_buffer(4096 + 64)
    base = (ctypes.addressof(buf) + 255) // 256 * 256
    return buf, [ctypes.c_void_p(base + 256 * i) for i in range(n)]


def test_verify_validation_errors(lib):
    keep, (q, kc, vc, kl, out, ws) = _fake(6)
    f = lib.sd_verify_attention
    args = dict(q=q, kc=kc, vc=vc, kl=kl, pt=None, mp=0, npg=0, lmax=64, out=out, lse=None,
                B=1, k=4, Hq=8, Hkv=2, D=128, scale=0.1, dt=1, ws=ws, wsb=1 << 30, st=None)

    def call(**kw):
        a = dict(args, **kw)
        return f(a["q"], a["kc"], a["vc"], a["kl"], a["pt"], a["mp"], a["npg"], a["lmax"],
                 a["out"], a["lse"], a["B"], a["k"], a["Hq"], a["Hkv"], a["D"], a["scale"],
                 a["dt"], a["ws"], a["wsb"], a["st"])

    assert call(q=None) == sd.SD_ERR_INVALID_ARG
    assert call(kl=None) == sd.SD_ERR_INVALID_ARG
    assert call(Hq=6, Hkv=4) == sd.SD_ERR_INVALID_ARG
    assert call(B=0) == sd.SD_ERR_INVALID_ARG
    assert call(dt=7) == sd.SD_ERR_INVALID_ARG
    assert call(scale=float("nan")) == sd.SD_ERR_INVALID_ARG
    assert call(lmax=0) == sd.SD_ERR_INVALID_ARG
    assert call(k=17) == sd.SD_ERR_UNSUPPORTED
    assert call(D=96) == sd.SD_ERR_UNSUPPORTED
    assert call(Hq=512, Hkv=1) == sd.SD_ERR_UNSUPPORTED
    assert call(dt=0, Hq=32, Hkv=1) == sd.SD_ERR_UNSUPPORTED   # fp32 path: <= 64 rows
    # bf16 tile list beyond 32-bit device indices: 4096 x 8 pairs x 2^15 tiles
    assert call(B=4096, Hq=8, Hkv=8, lmax=1 << 20) == sd.SD_ERR_UNSUPPORTED
    assert lib.sd_verify_workspace_size(4096, 4, 8, 8, 128, 1 << 20, 1) == 0
    # fp32: one work-group per (64-key split, sequence, KV head) below 2^31
    assert lib.sd_verify_workspace_size(1 << 20, 1, 1, 1, 64, 1 << 17, 0) == 0
    assert lib.sd_verify_workspace_size(1 << 10, 1, 1, 1, 64, 1 << 17, 0) > 0
    assert call(ws=None) == sd.SD_ERR_WORKSPACE
    assert call(wsb=16) == sd.SD_ERR_WORKSPACE
    # paged: needs a page count
    assert call(pt=kl, mp=0, npg=4) == sd.SD_ERR_INVALID_ARG
    assert call(pt=kl, mp=4, npg=0) == sd.SD_ERR_INVALID_ARG
    misaligned = ctypes.c_void_p(q.value + 2)
    assert call(q=misaligned) == sd.SD_ERR_INVALID_ARG


def test_compress_validation_errors(lib):
    keep, (lat, feats, out, ws) = _fake(4)
    f = lib.sd_latent_compress

    def call(lat=lat, feats=feats, out=out, B=1, N=64, C=16, d=256, H=2, scale=1.0, dt=1,
             ws=ws, wsb=1 << 30):
        return f(lat, feats, out, B, N, C, d, H, scale, dt, ws, wsb, None)

    assert call(lat=None) == sd.SD_ERR_INVALID_ARG
    assert call(N=0) == sd.SD_ERR_INVALID_ARG
    assert call(d=250, H=4) == sd.SD_ERR_INVALID_ARG
    assert call(scale=float("inf")) == sd.SD_ERR_INVALID_ARG
    assert call(d=96, H=1) == sd.SD_ERR_UNSUPPORTED
    assert call(d=1024, H=2) == sd.SD_ERR_UNSUPPORTED    # head width 512
    assert call(d=1024, H=2, dt=0) == sd.SD_ERR_UNSUPPORTED
    assert call(dt=2) == sd.SD_ERR_INVALID_ARG
    # feature rows wider than 2^22 channels (the copies' 24-bit row offsets)
    assert call(d=(1 << 22) + 128, H=(1 << 15) + 1) == sd.SD_ERR_UNSUPPORTED
    assert lib.sd_latent_compress_workspace_size(1, 64, 16, (1 << 22) + 128, (1 << 15) + 1, 1) == 0
    # bf16 with 256-channel heads: accepted, with one partial per short split
    assert lib.sd_latent_compress_workspace_size(1, 1000, 16, 512, 2, 1) > 0
    need = lib.sd_latent_compress_workspace_size(1, 65536, 16, 256, 2, 1)
    assert need > 0
    assert f(lat, feats, out, 1, 65536, 16, 256, 2, 1.0, 1, None, 0, None) == sd.SD_ERR_WORKSPACE


def test_accept_validation_errors(lib):
    keep, (p, q, d, u, n, t) = _fake(6)
    f = lib.sd_spec_accept

    def call(p=p, q=q, d=d, u=u, n=n, t=t, B=1, k=4, V=100, mode=1):
        return f(p, q, d, u, n, t, B, k, V, mode, None, 0, None)

    assert call(p=None) == sd.SD_ERR_INVALID_ARG
    assert call(q=None) == sd.SD_ERR_INVALID_ARG          # sampled needs q
    assert call(u=None) == sd.SD_ERR_INVALID_ARG
    assert call(mode=5) == sd.SD_ERR_INVALID_ARG
    assert call(V=0) == sd.SD_ERR_INVALID_ARG
    assert call(k=0) == sd.SD_ERR_INVALID_ARG
    assert call(k=17) == sd.SD_ERR_UNSUPPORTED
    assert call(V=(1 << 18) + 1) == sd.SD_ERR_UNSUPPORTED
    assert call(B=(1 << 22) + 1) == sd.SD_ERR_UNSUPPORTED    # grid bound
    assert lib.sd_spec_accept_workspace_size((1 << 22) + 1, 4, 100, 1) == 0
    assert lib.sd_spec_accept_workspace_size(1 << 22, 4, 100, 1) > 0
    assert lib.sd_spec_accept_logits_workspace_size((1 << 19) + 1, 4, 100, 1) == 0
    assert lib.sd_spec_accept_logits_workspace_size(1 << 19, 4, 100, 1) > 0


def test_accept_noalloc_validation_errors(lib):
    # the allocation-free acceptance checks everything before touching HIP:
    # invalid arguments, and shapes beyond its fixed 4 MiB scratch
    keep, (p, q, d, u, n, t) = _fake(6)
    f = lib.sd_spec_accept_noalloc

    def call(p=p, q=q, d=d, u=u, n=n, t=t, B=1, k=4, V=100, mode=1):
        return f(p, q, d, u, n, t, B, k, V, mode, None)

    assert call(p=None) == sd.SD_ERR_INVALID_ARG
    assert call(q=None) == sd.SD_ERR_INVALID_ARG
    assert call(n=None) == sd.SD_ERR_INVALID_ARG
    assert call(k=17) == sd.SD_ERR_UNSUPPORTED
    assert call(B=1025) == sd.SD_ERR_WORKSPACE             # more sequences than counters
    # greedy partials: 8 (k + 1) ceil(V / 1024) bytes per sequence, 34816 at
    # k = 16, V = 2^18: 121 sequences exceed 4 MiB - 4 KiB (120 would fit)
    assert call(B=121, k=16, V=1 << 18, mode=0) == sd.SD_ERR_WORKSPACE
    # sampled: 16 ceil(V / 1024) bytes per sequence, at most 4096 per
    # sequence, so 1024 sequences always fit


def test_compress_q8_validation_errors(lib):
    keep, (lq, le, fq, fe, out, ws) = _fake(6)
    f = lib.sd_latent_compress_q8

    def call(lq=lq, le=le, fq=fq, fe=fe, out=out, B=1, N=64, C=32, d=256, H=2, scale=1.0):
        return f(lq, le, fq, fe, out, B, N, C, d, H, scale, ws, 1 << 30, None)

    assert call(lq=None) == sd.SD_ERR_INVALID_ARG
    assert call(fe=None) == sd.SD_ERR_INVALID_ARG
    assert call(N=0) == sd.SD_ERR_INVALID_ARG
    assert call(d=255) == sd.SD_ERR_INVALID_ARG          # not a multiple of the heads
    assert call(H=4) == sd.SD_ERR_UNSUPPORTED             # 64-channel heads
    assert call(scale=float("nan")) == sd.SD_ERR_INVALID_ARG
    assert lib.sd_latent_compress_q8_workspace_size(1, 64, 32, 256, 4) == 0


def test_workspace_sizes_cover_the_partials(lib):
    # verify: one (D + 1)-float partial row per (sequence, KV head, split, row)
    for B, k, Hq, Hkv, D, cap in [(1, 4, 4, 1, 64, 608), (4, 8, 64, 8, 128, 65536),
                                  (16, 6, 32, 8, 128, 16384)]:
        for dt in (0, 1):
            if dt == 0 and k * Hq // Hkv > 64:
                continue
            n = lib.sd_verify_workspace_size(B, k, Hq, Hkv, D, cap, dt)
            assert n > 0 and n % 4 == 0
            assert n >= B * Hkv * k * (Hq // Hkv) * (D + 1) * 4
    assert lib.sd_verify_workspace_size(1, 4, 6, 4, 128, 100, 1) == 0   # invalid shape


def test_lm_head_validation_errors(lib):
    keep, (h, w, out, ws) = _fake(4)
    f = lib.sd_lm_head_probs

    def call(h=h, w=w, out=out, R=4, d=128, V=1000, tau=1.0, dt=1, ws=ws, wsb=1 << 30):
        return f(h, w, out, R, d, V, tau, dt, ws, wsb, None)

    assert call(h=None) == sd.SD_ERR_INVALID_ARG
    assert call(out=None) == sd.SD_ERR_INVALID_ARG
    assert call(R=0) == sd.SD_ERR_INVALID_ARG
    assert call(V=0) == sd.SD_ERR_INVALID_ARG
    assert call(tau=0.0) == sd.SD_ERR_INVALID_ARG
    assert call(tau=-1.0) == sd.SD_ERR_INVALID_ARG
    assert call(tau=float("nan")) == sd.SD_ERR_INVALID_ARG
    assert call(tau=float("inf")) == sd.SD_ERR_INVALID_ARG
    assert call(dt=3) == sd.SD_ERR_INVALID_ARG
    assert call(d=100) == sd.SD_ERR_UNSUPPORTED               # bf16: d % 64
    assert call(R=5000) == sd.SD_ERR_UNSUPPORTED
    assert call(R=257) == sd.SD_ERR_UNSUPPORTED                # bf16: one group of <= 16 row blocks
    assert call(R=257, dt=0) != sd.SD_ERR_UNSUPPORTED
    assert call(h=ctypes.c_void_p(h.value + 8)) == sd.SD_ERR_INVALID_ARG   # bf16: 16-byte aligned
    assert call(ws=None) == sd.SD_ERR_WORKSPACE
    assert call(wsb=8) == sd.SD_ERR_WORKSPACE
    # block (max, sum) pairs of 16 entries per row, then one pair per row
    n = lib.sd_lm_head_workspace_size(36, 8192, 152064, 1)
    assert n == (36 * (152064 // 16) + 36) * 8
    assert lib.sd_lm_head_workspace_size(0, 64, 10, 1) == 0


def test_sample_validation_errors(lib):
    keep, (p, u, t, ws) = _fake(4)
    f = lib.sd_sample_tokens

    def call(p=p, u=u, t=t, R=3, V=100, ws=ws, wsb=1 << 30):
        return f(p, u, t, R, V, ws, wsb, None)

    assert call(p=None) == sd.SD_ERR_INVALID_ARG
    assert call(u=None) == sd.SD_ERR_INVALID_ARG
    assert call(t=None) == sd.SD_ERR_INVALID_ARG
    assert call(R=0) == sd.SD_ERR_INVALID_ARG
    assert call(V=(1 << 18) + 1) == sd.SD_ERR_UNSUPPORTED
    assert call(ws=None) == sd.SD_ERR_WORKSPACE
    assert call(wsb=lib.sd_sample_workspace_size(3, 100) - 1) == sd.SD_ERR_WORKSPACE
    assert lib.sd_sample_workspace_size(3, 100) >= 3 * 4


def test_accept_logits_validation_errors(lib):
    keep, (zt, zd, d, n, t, ws) = _fake(6)
    f = lib.sd_spec_accept_logits

    def call(zt=zt, zd=zd, d=d, n=n, t=t, tau=0.7, B=1, k=4, V=100, dt=0, mode=1, ws=ws, wsb=1 << 30):
        return f(zt, zd, d, 1, 2, tau, n, t, B, k, V, dt, mode, ws, wsb, None)

    assert call(zt=None) == sd.SD_ERR_INVALID_ARG
    assert call(zd=None) == sd.SD_ERR_INVALID_ARG         # sampled needs draft logits
    assert call(tau=0.0) == sd.SD_ERR_INVALID_ARG
    assert call(tau=float("nan")) == sd.SD_ERR_INVALID_ARG
    assert call(dt=3) == sd.SD_ERR_INVALID_ARG
    assert call(mode=4) == sd.SD_ERR_INVALID_ARG
    assert call(B=0) == sd.SD_ERR_INVALID_ARG
    assert call(k=17) == sd.SD_ERR_UNSUPPORTED
    assert call(V=(1 << 18) + 1) == sd.SD_ERR_UNSUPPORTED
    assert call(ws=None) == sd.SD_ERR_WORKSPACE
    assert call(wsb=16) == sd.SD_ERR_WORKSPACE
    # the sampled workspace adds the logits' row statistics to the rule's
    greedy = lib.sd_spec_accept_logits_workspace_size(4, 8, 152064, 0)
    sampled = lib.sd_spec_accept_logits_workspace_size(4, 8, 152064, 1)
    assert sampled >= lib.sd_spec_accept_workspace_size(4, 8, 152064, 1) + 4 * 17 * 38 * 8
    assert greedy == lib.sd_spec_accept_workspace_size(4, 8, 152064, 0)
    assert lib.sd_spec_accept_logits_workspace_size(4, 17, 100, 1) == 0

    g = lib.sd_philox_uniforms
    assert g(1, 2, None, 1, 4, None) == sd.SD_ERR_INVALID_ARG
    assert g(1, 2, n, 0, 4, None) == sd.SD_ERR_INVALID_ARG
    assert g(1, 2, n, 1, 0, None) == sd.SD_ERR_INVALID_ARG
    assert g(1, 2, n, 1, (1 << 16) + 1, None) == sd.SD_ERR_UNSUPPORTED


def test_linear_validation_errors(lib):
    # every call below fails validation, so nothing is launched
    keep, (x, w, b, r, y, ws) = _fake(6)
    f = lib.sd_linear

    def call(x=x, w=w, b=None, r=None, y=y, R=4, K=512, N=100, ws=ws, wsb=0):
        return f(x, w, b, r, y, R, K, N, ws, wsb, None)

    assert call(x=None) == sd.SD_ERR_INVALID_ARG
    assert call(y=None) == sd.SD_ERR_INVALID_ARG
    assert call(R=0) == sd.SD_ERR_INVALID_ARG
    assert call(N=0) == sd.SD_ERR_INVALID_ARG
    assert call(K=300) == sd.SD_ERR_UNSUPPORTED                # K % 256
    assert call(K=128) == sd.SD_ERR_UNSUPPORTED
    assert call(R=1 << 16, N=1 << 16) == sd.SD_ERR_UNSUPPORTED  # R * N > 2^31
    assert call(x=ctypes.c_void_p(x.value + 8)) == sd.SD_ERR_INVALID_ARG
    assert call(ws=None) == sd.SD_ERR_WORKSPACE
    assert call(wsb=8) == sd.SD_ERR_WORKSPACE
    # one fp32 partial per reduction split; at most 16 splits
    n = lib.sd_linear_workspace_size(36, 8192, 8192)
    assert n >= 36 * 8192 * 4 and n % (36 * 8192 * 4) == 0 and n <= 16 * 36 * 8192 * 4
    assert lib.sd_linear_workspace_size(36, 300, 10) == 0


def test_semi_ar_layer_validation_errors(lib):
    keep, ptrs = _fake(14)
    f = lib.sd_semi_ar_layer
    P = dict(zip(["u", "fcw", "fcb", "ln1", "wqkv", "wo", "ln2", "wgu", "wdown", "kc", "vc", "pos", "out",
                  "ws"], ptrs))

    def call(B=2, r=9, d=1024, hq=8, hkv=2, I=2048, L=64, eps=1e-6, theta=1e4, wsb=0, **kw):
        p = dict(P, **kw)
        return f(p["u"], p["fcw"], p["fcb"], p["ln1"], p["wqkv"], p["wo"], p["ln2"], p["wgu"], p["wdown"],
                 p["kc"], p["vc"], p["pos"], p["out"], B, r, d, hq, hkv, I, L, eps, theta, p["ws"], wsb, None)

    assert call(u=None) == sd.SD_ERR_INVALID_ARG
    assert call(pos=None) == sd.SD_ERR_INVALID_ARG
    assert call(B=0) == sd.SD_ERR_INVALID_ARG
    assert call(hq=3) == sd.SD_ERR_INVALID_ARG                  # d % hq
    assert call(hkv=3) == sd.SD_ERR_INVALID_ARG                 # hq % hkv
    assert call(r=17) == sd.SD_ERR_UNSUPPORTED
    assert call(d=1024, hq=4) == sd.SD_ERR_UNSUPPORTED          # D = 256
    assert call(I=1000) == sd.SD_ERR_UNSUPPORTED                # I % 256
    assert call(L=8) == sd.SD_ERR_UNSUPPORTED                   # Lmax < r
    assert call(eps=-1.0) == sd.SD_ERR_INVALID_ARG
    assert call(theta=0.0) == sd.SD_ERR_INVALID_ARG
    assert call(theta=float("nan")) == sd.SD_ERR_INVALID_ARG
    assert call(wgu=ctypes.c_void_p(ptrs[7].value + 8)) == sd.SD_ERR_INVALID_ARG
    assert call(ws=None) == sd.SD_ERR_WORKSPACE
    assert call(wsb=64) == sd.SD_ERR_WORKSPACE
    assert lib.sd_semi_ar_layer_workspace_size(2, 9, 1024, 8, 2, 2048, 64) > 2 * 9 * 2048 * 2
    assert lib.sd_semi_ar_layer_workspace_size(2, 17, 1024, 8, 2, 2048, 64) == 0


def test_semi_ar_draft_validation_errors(lib):
    keep, ptrs = _fake(15)
    f = lib.sd_semi_ar_draft
    names = ["u0", "fcw", "fcb", "ln1", "wqkv", "wo", "ln2", "wgu", "wdown", "lmw", "emb", "ph", "kc", "vc",
             "pos"]
    P = dict(zip(names, ptrs))
    keep2, (uu, tok, q, ws) = _fake(4)
    P.update(u=uu, tok=tok, q=q, ws=ws)

    def call(B=2, r0=3, d=1024, hq=8, hkv=2, I=2048, L=64, V=1000, K=6, kp=2, eps=1e-6, theta=1e4, tau=0.8,
             wsb=0, **kw):
        p = dict(P, **kw)
        return f(*[p[n] for n in names], p["u"], p["tok"], p["q"], B, r0, d, hq, hkv, I, L, V, K, kp, eps, theta,
                 tau, p["ws"], wsb, None)

    assert call(lmw=None) == sd.SD_ERR_INVALID_ARG
    assert call(q=None) == sd.SD_ERR_INVALID_ARG
    assert call(K=5) == sd.SD_ERR_INVALID_ARG                  # K % k'
    assert call(kp=4) == sd.SD_ERR_INVALID_ARG                 # k' > r0
    assert call(kp=0) == sd.SD_ERR_INVALID_ARG
    assert call(r0=12, kp=9, K=9) == sd.SD_ERR_UNSUPPORTED     # k' > 8
    assert call(V=(1 << 18) + 1) == sd.SD_ERR_UNSUPPORTED
    assert call(B=200, kp=2) == sd.SD_ERR_UNSUPPORTED          # B k' > 256
    assert call(tau=0.0) == sd.SD_ERR_INVALID_ARG
    assert call(ws=None) == sd.SD_ERR_WORKSPACE
    assert lib.sd_semi_ar_draft_workspace_size(2, 3, 1024, 8, 2, 2048, 64, 1000, 6, 2) > 0
    assert lib.sd_semi_ar_draft_workspace_size(2, 3, 1024, 8, 2, 2048, 64, 1000, 5, 2) == 0


def test_q8_validation_errors(lib):
    keep, (x, w, s, y, ws) = _fake(5)
    f = lib.sd_linear_q8

    def call(x=x, w=w, s=s, y=y, R=4, K=512, N=100, ws=ws, wsb=0):
        return f(x, w, s, None, None, y, R, K, N, ws, wsb, None)

    assert call(s=None) == sd.SD_ERR_INVALID_ARG
    assert call(w=None) == sd.SD_ERR_INVALID_ARG
    assert call(K=300) == sd.SD_ERR_UNSUPPORTED
    assert call(w=ctypes.c_void_p(w.value + 8)) == sd.SD_ERR_INVALID_ARG
    assert call(wsb=8) == sd.SD_ERR_WORKSPACE
    keep2, ptrs = _fake(18)
    g = lib.sd_semi_ar_layer_q8

    def lcall(r=9, wgu_s=ptrs[11], ws=ptrs[17], wsb=0):
        # u, fc_w, fc_s, fc_b, ln1, wqkv, wqkv_s, wo, wo_s, ln2, wgu, wgu_s,
        # wdown, wdown_s, k_cache, v_cache, pos, out
        p = list(ptrs[:18])
        p[11] = wgu_s
        return g(*p, 2, r, 1024, 8, 2, 2048, 64, 1e-6, 1e4, ws, wsb, None)

    assert lcall(wgu_s=None) == sd.SD_ERR_INVALID_ARG
    assert lcall(r=17) == sd.SD_ERR_UNSUPPORTED
    assert lcall(ws=None) == sd.SD_ERR_WORKSPACE


def test_avg_pool_validation_errors(lib):
    keep, (f, o) = _fake(2)
    call = lambda B=2, N=16, C=4, d=64, dt=1, f=f, o=o: lib.sd_avg_pool_compress(f, o, B, N, C, d, dt, None)
    assert call(C=17) == sd.SD_ERR_INVALID_ARG                  # C > N
    assert call(C=0) == sd.SD_ERR_INVALID_ARG
    assert call(dt=2) == sd.SD_ERR_INVALID_ARG
    assert call(f=None) == sd.SD_ERR_INVALID_ARG
    assert call(N=1 << 25, C=70000) == sd.SD_ERR_UNSUPPORTED
