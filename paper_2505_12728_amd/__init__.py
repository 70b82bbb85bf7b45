"""SpecFLASH draft-verify hot path on MI355X: Python binding of libspecflash.

The three entry points mirror the C ABI in include/specflash.h and only
marshal arguments: every step of the computation runs in the HIP kernels of
libspecflash.so (built by ``paper_2505_12728_amd.build``).  torch supplies
device memory and the current HIP stream.  There is no fallback: if the
library is missing or the tensors are not on the GPU, the calls raise.

    sd_latent_compress   Sec. 3.2, Eq. 3 (learned queries attend over F_V)
    sd_verify_attention  Sec. 3.1 (one parallel pass over the K drafts)
    sd_spec_accept       Sec. 3.1 / 3.3 acceptance; greedy for Sec. 4.2
    sd_lm_head_probs     Sec. 3.1 / 3.3, Algorithm 1: LM head + softmax(z / tau)
    sd_sample_tokens     Algorithm 1: drafts drawn from their distributions
"""

import ctypes
import math
import os

__all__ = [
    "SD_OK", "SD_ERR_INVALID_ARG", "SD_ERR_UNSUPPORTED", "SD_ERR_WORKSPACE", "SD_ERR_HIP",
    "SD_F32", "SD_BF16", "SD_ACCEPT_GREEDY", "SD_ACCEPT_SAMPLED",
    "SDError", "library", "library_path",
    "sd_status_string", "sd_version",
    "sd_latent_compress_workspace_size", "sd_latent_compress",
    "sd_verify_workspace_size", "sd_verify_attention",
    "sd_spec_accept_workspace_size", "sd_spec_accept", "sd_spec_accept_noalloc",
    "sd_lm_head_workspace_size", "sd_lm_head_probs",
    "sd_sample_workspace_size", "sd_sample_tokens",
    "sd_spec_accept_logits_workspace_size", "sd_spec_accept_logits", "sd_philox_uniforms",
    "sd_linear_workspace_size", "sd_linear",
    "sd_semi_ar_layer_workspace_size", "sd_semi_ar_layer",
    "sd_semi_ar_draft_workspace_size", "sd_semi_ar_draft",
    "sd_linear_q8", "sd_semi_ar_layer_q8", "sd_avg_pool_compress",
    "sd_latent_compress_q8_workspace_size", "sd_latent_compress_q8",
]

SD_OK, SD_ERR_INVALID_ARG, SD_ERR_UNSUPPORTED, SD_ERR_WORKSPACE, SD_ERR_HIP = 0, 1, 2, 3, 4
SD_F32, SD_BF16 = 0, 1
SD_ACCEPT_GREEDY, SD_ACCEPT_SAMPLED = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libspecflash.so")
_lib = None

_c = ctypes
_vp, _sz, _i, _f = _c.c_void_p, _c.c_size_t, _c.c_int, _c.c_float
_SIGNATURES = {
    "sd_status_string": (_c.c_char_p, [_i]),
    "sd_version": (_i, []),
    "sd_latent_compress_workspace_size": (_sz, [_i, _i, _i, _i, _i, _i]),
    "sd_latent_compress": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _f, _i, _vp, _sz, _vp]),
    "sd_verify_workspace_size": (_sz, [_i, _i, _i, _i, _i, _i, _i]),
    "sd_verify_attention": (_i, [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _vp, _vp,
                                 _i, _i, _i, _i, _i, _f, _i, _vp, _sz, _vp]),
    "sd_spec_accept_workspace_size": (_sz, [_i, _i, _i, _i]),
    "sd_spec_accept": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp, _sz, _vp]),
    "sd_spec_accept_noalloc": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp]),
    "sd_spec_accept_logits_workspace_size": (_sz, [_i, _i, _i, _i]),
    "sd_spec_accept_logits": (_i, [_vp, _vp, _vp, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_float,
                                   _vp, _vp, _i, _i, _i, _i, _i, _vp, _sz, _vp]),
    "sd_philox_uniforms": (_i, [ctypes.c_uint64, ctypes.c_uint64, _vp, _i, _i, _vp]),
    "sd_lm_head_workspace_size": (_sz, [_i, _i, _i, _i]),
    "sd_lm_head_probs": (_i, [_vp, _vp, _vp, _i, _i, _i, _f, _i, _vp, _sz, _vp]),
    "sd_sample_workspace_size": (_sz, [_i, _i]),
    "sd_sample_tokens": (_i, [_vp, _vp, _vp, _i, _i, _vp, _sz, _vp]),
    "sd_linear_workspace_size": (_sz, [_i, _i, _i]),
    "sd_linear": (_i, [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _vp, _sz, _vp]),
    "sd_semi_ar_layer_workspace_size": (_sz, [_i, _i, _i, _i, _i, _i, _i]),
    "sd_semi_ar_layer": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                              _i, _i, _i, _i, _i, _i, _i, _f, _f, _vp, _sz, _vp]),
    "sd_semi_ar_draft_workspace_size": (_sz, [_i] * 10),
    "sd_linear_q8": (_i, [_vp] * 6 + [_i, _i, _i, _vp, _sz, _vp]),
    "sd_avg_pool_compress": (_i, [_vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "sd_latent_compress_q8_workspace_size": (_sz, [_i, _i, _i, _i, _i]),
    "sd_latent_compress_q8": (_i, [_vp] * 5 + [_i] * 5 + [_f, _vp, _sz, _vp]),
    "sd_semi_ar_layer_q8": (_i, [_vp] * 18 + [_i] * 7 + [_f, _f, _vp, _sz, _vp]),
    "sd_semi_ar_draft": (_i, [_vp] * 18 + [_i] * 10 + [_f, _f, _f, _vp, _sz, _vp]),
}


class SDError(RuntimeError):
    """A non-zero sd_status returned by the library."""

    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {sd_status_string(status)}")


def library():
    """Load libspecflash.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(library_path):
            raise RuntimeError(
                f"{library_path} is missing: build it with `python -m paper_2505_12728_amd.build`")
        lib = ctypes.CDLL(library_path)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def sd_status_string(status):
    return library().sd_status_string(int(status)).decode()


def sd_version():
    return library().sd_version()


# ----------------------------------------------------------------- helpers

def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return SD_F32
    if t.dtype == torch.bfloat16:
        return SD_BF16
    raise TypeError(f"unsupported dtype {t.dtype}: use float32 or bfloat16")


def _check(t, name, dtype=None, ndim=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got {t.dim()}")


def _out(t, name, shape, dtype, device):
    """A caller-supplied output (or workspace) must be a contiguous tensor of
    exactly the expected shape and dtype on the inputs' device: the kernels
    write its whole extent, so a short buffer would be overrun on the device."""
    _check(t, name, dtype=dtype)
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    return t


def _same_device(name, t, device):
    if t is not None and t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _workspace(nbytes, device, given):
    if nbytes == 0:
        return None, 0
    if given is not None:
        _check(given, "workspace")
        _same_device("workspace", given, device)
        return given, given.numel() * given.element_size()
    torch = _torch()
    # zero-filled: some entry points keep arrival counters in the workspace
    # that must start at zero (every call returns them to zero)
    return torch.zeros(nbytes, dtype=torch.uint8, device=device), nbytes


def _raise(status, where):
    if status != SD_OK:
        raise SDError(status, where)


# ------------------------------------------------------------- compression

def sd_latent_compress_workspace_size(B, N, C, d, num_heads, dtype):
    return library().sd_latent_compress_workspace_size(B, N, C, d, num_heads, dtype)


def sd_latent_compress(latents, feats, num_heads=1, scale=1.0, out=None, workspace=None,
                       stream=None):
    """Eq. 3 per head slice: latents [C, d], feats [B, N, d] -> out [B, C, d] fp32."""
    torch = _torch()
    _check(latents, "latents", ndim=2)
    _check(feats, "feats", dtype=latents.dtype, ndim=3)
    C, d = latents.shape
    B, N, d2 = feats.shape
    if d2 != d:
        raise ValueError("latents and feats disagree on the feature width")
    dt = _dtype_code(latents)
    _same_device("feats", feats, latents.device)
    if out is None:
        out = torch.empty((B, C, d), dtype=torch.float32, device=feats.device)
    _out(out, "out", (B, C, d), torch.float32, feats.device)
    ws_bytes = sd_latent_compress_workspace_size(B, N, C, d, num_heads, dt)
    ws, ws_len = _workspace(ws_bytes, feats.device, workspace)
    st = library().sd_latent_compress(_ptr(latents), _ptr(feats), _ptr(out), B, N, C, d,
                                      num_heads, float(scale), dt, _ptr(ws), ws_len,
                                      _stream(stream))
    _raise(st, "sd_latent_compress")
    return out


def sd_latent_compress_q8_workspace_size(B, N, C, d, num_heads):
    return library().sd_latent_compress_q8_workspace_size(B, N, C, d, num_heads)


def sd_latent_compress_q8(latents_q, latent_exp, feats_q, feat_exp, num_heads=1, scale=1.0, out=None,
                          workspace=None, stream=None):
    """Eq. 3 on int8 rows with power-of-two row scales: latents_q [C, d] int8
    with latent_exp [C] int8, feats_q [B, N, d] int8 with feat_exp [B, N]
    int8 (row r stands for q[r] * 2^e[r]).  Returns out [B, C, d] fp32."""
    torch = _torch()
    _check(latents_q, "latents_q", dtype=torch.int8, ndim=2)
    _check(feats_q, "feats_q", dtype=torch.int8, ndim=3)
    _check(latent_exp, "latent_exp", dtype=torch.int8, ndim=1)
    _check(feat_exp, "feat_exp", dtype=torch.int8, ndim=2)
    C, d = latents_q.shape
    B, N, d2 = feats_q.shape
    if d2 != d or latent_exp.shape[0] != C or tuple(feat_exp.shape) != (B, N):
        raise ValueError("latents_q [C, d], latent_exp [C], feats_q [B, N, d], feat_exp [B, N] expected")
    dev = feats_q.device
    for name, t in (("latents_q", latents_q), ("latent_exp", latent_exp), ("feat_exp", feat_exp)):
        _same_device(name, t, dev)
    if out is None:
        out = torch.empty((B, C, d), dtype=torch.float32, device=dev)
    _out(out, "out", (B, C, d), torch.float32, dev)
    ws_bytes = sd_latent_compress_q8_workspace_size(B, N, C, d, num_heads)
    ws, ws_len = _workspace(ws_bytes, dev, workspace)
    st = library().sd_latent_compress_q8(_ptr(latents_q), _ptr(latent_exp), _ptr(feats_q), _ptr(feat_exp),
                                         _ptr(out), B, N, C, d, num_heads, float(scale), _ptr(ws), ws_len,
                                         _stream(stream))
    _raise(st, "sd_latent_compress_q8")
    return out


# ------------------------------------------------------------ verification

def sd_verify_workspace_size(B, k, Hq, Hkv, D, capacity, dtype):
    return library().sd_verify_workspace_size(B, k, Hq, Hkv, D, capacity, dtype)


def sd_verify_attention(q, k_cache, v_cache, kv_len, scale=None, page_table=None,
                        num_pages=None, out=None, lse=True, workspace=None, stream=None):
    """Attention of the k block queries over the cache (causal inside the block).

    q [B, k, Hq, D]; caches [B, Lmax, Hkv, D], or page pools [P, Hkv, 16, D]
    with page_table [B, max_pages] int32; kv_len [B] int32 (block included).
    Returns (out [B, k, Hq, D] fp32, lse [B, k, Hq] fp32 or None).
    ``scale`` multiplies q . k; the paper names no scale, and None passes the
    standard attention scale 1 / sqrt(D) to the library explicitly (the C
    entry point itself takes the scale as a required argument).
    """
    torch = _torch()
    _check(q, "q", ndim=4)
    _check(k_cache, "k_cache", dtype=q.dtype, ndim=4)
    _check(v_cache, "v_cache", dtype=q.dtype, ndim=4)
    _check(kv_len, "kv_len", dtype=torch.int32, ndim=1)
    B, k, Hq, D = q.shape
    if tuple(k_cache.shape) != tuple(v_cache.shape):
        raise ValueError("k_cache and v_cache must have the same shape")
    if kv_len.shape[0] != B:
        raise ValueError("kv_len needs one entry per sequence")
    dt = _dtype_code(q)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if page_table is None:
        if k_cache.shape[0] != B or k_cache.shape[3] != D:
            raise ValueError("contiguous caches must be [B, Lmax, Hkv, D]")
        Lmax, Hkv = k_cache.shape[1], k_cache.shape[2]
        max_pages = num_pages_ = 0
        capacity = Lmax
    else:
        _check(page_table, "page_table", dtype=torch.int32, ndim=2)
        if k_cache.shape[2] != 16 or k_cache.shape[3] != D or page_table.shape[0] != B:
            raise ValueError("paged caches must be [P, Hkv, 16, D] with a [B, max_pages] table")
        Hkv = k_cache.shape[1]
        max_pages = page_table.shape[1]
        num_pages_ = k_cache.shape[0] if num_pages is None else num_pages
        Lmax = 0
        capacity = 16 * max_pages
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("kv_len", kv_len),
                    ("page_table", page_table)):
        _same_device(name, t, q.device)
    if out is None:
        out = torch.empty((B, k, Hq, D), dtype=torch.float32, device=q.device)
    _out(out, "out", (B, k, Hq, D), torch.float32, q.device)
    lse_t = None
    if lse is True:
        lse_t = torch.empty((B, k, Hq), dtype=torch.float32, device=q.device)
    elif lse is not None and lse is not False:
        lse_t = _out(lse, "lse", (B, k, Hq), torch.float32, q.device)
    ws_bytes = sd_verify_workspace_size(B, k, Hq, Hkv, D, capacity, dt)
    ws, ws_len = _workspace(ws_bytes, q.device, workspace)
    st = library().sd_verify_attention(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(kv_len),
                                       _ptr(page_table), max_pages, num_pages_, Lmax, _ptr(out),
                                       _ptr(lse_t), B, k, Hq, Hkv, D, float(scale), dt,
                                       _ptr(ws), ws_len, _stream(stream))
    _raise(st, "sd_verify_attention")
    return out, lse_t


# -------------------------------------------------------------- acceptance

def sd_spec_accept_workspace_size(B, k, V, mode):
    return library().sd_spec_accept_workspace_size(B, k, V, mode)


def sd_spec_accept(p, q, draft, u, mode=SD_ACCEPT_SAMPLED, n_accepted=None, tokens=None,
                   workspace=None, stream=None):
    """Speculative acceptance: p [B, k+1, V], q [B, k, V], draft [B, k] int32,
    u [B, k+1] fp32.  Returns (n_accepted [B] int32, tokens [B, k+1] int32)."""
    torch = _torch()
    _check(p, "p", dtype=torch.float32, ndim=3)
    _check(draft, "draft", dtype=torch.int32, ndim=2)
    B, kp1, V = p.shape
    k = kp1 - 1
    if tuple(draft.shape) != (B, k):
        raise ValueError("draft must be [B, k]")
    if mode == SD_ACCEPT_SAMPLED:
        _check(q, "q", dtype=torch.float32, ndim=3)
        _check(u, "u", dtype=torch.float32, ndim=2)
        if tuple(q.shape) != (B, k, V) or tuple(u.shape) != (B, k + 1):
            raise ValueError("q must be [B, k, V] and u [B, k+1]")
    for name, t in (("q", q if mode == SD_ACCEPT_SAMPLED else None), ("draft", draft),
                    ("u", u if mode == SD_ACCEPT_SAMPLED else None)):
        _same_device(name, t, p.device)
    if n_accepted is None:
        n_accepted = torch.empty((B,), dtype=torch.int32, device=p.device)
    if tokens is None:
        tokens = torch.empty((B, k + 1), dtype=torch.int32, device=p.device)
    _out(n_accepted, "n_accepted", (B,), torch.int32, p.device)
    _out(tokens, "tokens", (B, k + 1), torch.int32, p.device)
    ws_bytes = sd_spec_accept_workspace_size(B, k, V, mode)
    ws, ws_len = _workspace(ws_bytes, p.device, workspace)
    st = library().sd_spec_accept(_ptr(p), _ptr(q), _ptr(draft), _ptr(u), _ptr(n_accepted),
                                  _ptr(tokens), B, k, V, int(mode), _ptr(ws), ws_len,
                                  _stream(stream))
    _raise(st, "sd_spec_accept")
    return n_accepted, tokens


def sd_spec_accept_noalloc(p, q, draft, u, mode=SD_ACCEPT_SAMPLED, n_accepted=None, tokens=None,
                           stream=None):
    """sd_spec_accept with the library's fixed device scratch instead of a
    workspace (for callers that cannot allocate; pass n_accepted and tokens
    to allocate nothing here either).  Same arguments and results."""
    torch = _torch()
    _check(p, "p", dtype=torch.float32, ndim=3)
    _check(draft, "draft", dtype=torch.int32, ndim=2)
    B, kp1, V = p.shape
    k = kp1 - 1
    if tuple(draft.shape) != (B, k):
        raise ValueError("draft must be [B, k]")
    if mode == SD_ACCEPT_SAMPLED:
        _check(q, "q", dtype=torch.float32, ndim=3)
        _check(u, "u", dtype=torch.float32, ndim=2)
        if tuple(q.shape) != (B, k, V) or tuple(u.shape) != (B, k + 1):
            raise ValueError("q must be [B, k, V] and u [B, k+1]")
        _same_device("q", q, p.device)
        _same_device("u", u, p.device)
    _same_device("draft", draft, p.device)
    if n_accepted is None:
        n_accepted = torch.empty((B,), dtype=torch.int32, device=p.device)
    if tokens is None:
        tokens = torch.empty((B, k + 1), dtype=torch.int32, device=p.device)
    _out(n_accepted, "n_accepted", (B,), torch.int32, p.device)
    _out(tokens, "tokens", (B, k + 1), torch.int32, p.device)
    st = library().sd_spec_accept_noalloc(_ptr(p), _ptr(q), _ptr(draft), _ptr(u), _ptr(n_accepted),
                                          _ptr(tokens), B, k, V, int(mode), _stream(stream))
    _raise(st, "sd_spec_accept_noalloc")
    return n_accepted, tokens


def sd_spec_accept_logits_workspace_size(B, k, V, mode):
    return library().sd_spec_accept_logits_workspace_size(B, k, V, mode)


def sd_spec_accept_logits(target_logits, draft_logits, draft, seed, offset, temperature,
                          mode=SD_ACCEPT_SAMPLED, n_accepted=None, tokens=None, workspace=None,
                          stream=None):
    """Acceptance from logits: target_logits [B, k+1, V], draft_logits [B, k, V]
    (fp32 or bf16, same dtype), draft [B, k] int32; uniforms from Philox(seed,
    offset).  Returns (n_accepted [B] int32, tokens [B, k+1] int32)."""
    torch = _torch()
    _check(target_logits, "target_logits", ndim=3)
    _check(draft, "draft", dtype=torch.int32, ndim=2)
    B, kp1, V = target_logits.shape
    k = kp1 - 1
    if tuple(draft.shape) != (B, k):
        raise ValueError("draft must be [B, k]")
    if mode == SD_ACCEPT_SAMPLED:
        _check(draft_logits, "draft_logits", dtype=target_logits.dtype, ndim=3)
        if tuple(draft_logits.shape) != (B, k, V):
            raise ValueError("draft_logits must be [B, k, V]")
    dt = _dtype_code(target_logits)
    dev = target_logits.device
    _same_device("draft", draft, dev)
    if mode == SD_ACCEPT_SAMPLED:
        _same_device("draft_logits", draft_logits, dev)
    if n_accepted is None:
        n_accepted = torch.empty((B,), dtype=torch.int32, device=dev)
    if tokens is None:
        tokens = torch.empty((B, k + 1), dtype=torch.int32, device=dev)
    _out(n_accepted, "n_accepted", (B,), torch.int32, dev)
    _out(tokens, "tokens", (B, k + 1), torch.int32, dev)
    ws_bytes = sd_spec_accept_logits_workspace_size(B, k, V, mode)
    ws, ws_len = _workspace(ws_bytes, target_logits.device, workspace)
    st = library().sd_spec_accept_logits(_ptr(target_logits), _ptr(draft_logits), _ptr(draft),
                                         int(seed), int(offset), float(temperature),
                                         _ptr(n_accepted), _ptr(tokens), B, k, V, dt, int(mode),
                                         _ptr(ws), ws_len, _stream(stream))
    _raise(st, "sd_spec_accept_logits")
    return n_accepted, tokens


def sd_philox_uniforms(seed, offset, B, n, out=None, device=None, stream=None):
    """u [B, n] float32 on the device: the acceptance uniforms of (seed, offset)."""
    torch = _torch()
    if out is None:
        out = torch.empty((B, n), dtype=torch.float32, device=device or "cuda")
    _out(out, "out", (B, n), torch.float32, out.device)
    st = library().sd_philox_uniforms(int(seed), int(offset), _ptr(out), B, n, _stream(stream))
    _raise(st, "sd_philox_uniforms")
    return out


def sd_lm_head_workspace_size(R, d, V, dtype):
    return library().sd_lm_head_workspace_size(R, d, V, dtype)


def sd_lm_head_probs(hidden, weight, temperature, out=None, workspace=None, stream=None):
    """LM head + temperature softmax: hidden [R, d], weight [V, d] (bf16 or
    fp32, same dtype).  Returns probs [R, V] fp32 = softmax(hidden W^T / tau)."""
    torch = _torch()
    _check(hidden, "hidden", ndim=2)
    _check(weight, "weight", dtype=hidden.dtype, ndim=2)
    R, d = hidden.shape
    V = weight.shape[0]
    if weight.shape[1] != d:
        raise ValueError("weight must be [V, d] with the hidden width d")
    dt = _dtype_code(hidden)
    _same_device("weight", weight, hidden.device)
    if out is None:
        out = torch.empty((R, V), dtype=torch.float32, device=hidden.device)
    _out(out, "out", (R, V), torch.float32, hidden.device)
    ws_bytes = sd_lm_head_workspace_size(R, d, V, dt)
    ws, ws_len = _workspace(ws_bytes, hidden.device, workspace)
    st = library().sd_lm_head_probs(_ptr(hidden), _ptr(weight), _ptr(out), R, d, V,
                                    float(temperature), dt, _ptr(ws), ws_len, _stream(stream))
    _raise(st, "sd_lm_head_probs")
    return out


def sd_sample_workspace_size(R, V):
    return library().sd_sample_workspace_size(R, V)


def sd_sample_tokens(probs, u, out=None, workspace=None, stream=None):
    """T_r ~ Categorical(probs[r]) (exact fixed-point inverse CDF): probs [R, V]
    fp32, u [R] fp32.  Returns tokens [R] int32."""
    torch = _torch()
    _check(probs, "probs", dtype=torch.float32, ndim=2)
    _check(u, "u", dtype=torch.float32, ndim=1)
    R, V = probs.shape
    if u.shape[0] != R:
        raise ValueError("u must be [R]")
    _same_device("u", u, probs.device)
    if out is None:
        out = torch.empty((R,), dtype=torch.int32, device=probs.device)
    _out(out, "out", (R,), torch.int32, probs.device)
    ws_bytes = sd_sample_workspace_size(R, V)
    ws, ws_len = _workspace(ws_bytes, probs.device, workspace)
    st = library().sd_sample_tokens(_ptr(probs), _ptr(u), _ptr(out), R, V, _ptr(ws), ws_len,
                                    _stream(stream))
    _raise(st, "sd_sample_tokens")
    return out


def sd_linear_workspace_size(R, K, N):
    return library().sd_linear_workspace_size(R, K, N)


def sd_linear(x, w, bias=None, residual=None, out=None, workspace=None, stream=None):
    """y = x W^T (+ bias) (+ residual): x [R, K] bf16, w [N, K] bf16, bias [N]
    fp32, residual [R, N] fp32.  Returns y [R, N] fp32."""
    torch = _torch()
    _check(x, "x", dtype=torch.bfloat16, ndim=2)
    _check(w, "w", dtype=torch.bfloat16, ndim=2)
    R, K = x.shape
    N = w.shape[0]
    if w.shape[1] != K:
        raise ValueError("w must be [N, K] with the width K of x")
    if bias is not None:
        _check(bias, "bias", dtype=torch.float32, ndim=1)
        if bias.shape[0] != N:
            raise ValueError("bias must be [N]")
    if residual is not None:
        _check(residual, "residual", dtype=torch.float32, ndim=2)
        if tuple(residual.shape) != (R, N):
            raise ValueError("residual must be [R, N]")
    for name, t in (("w", w), ("bias", bias), ("residual", residual)):
        _same_device(name, t, x.device)
    if out is None:
        out = torch.empty((R, N), dtype=torch.float32, device=x.device)
    _out(out, "out", (R, N), torch.float32, x.device)
    ws_bytes = sd_linear_workspace_size(R, K, N)
    ws, ws_len = _workspace(ws_bytes, x.device, workspace)
    st = library().sd_linear(_ptr(x), _ptr(w), _ptr(bias), _ptr(residual), _ptr(out), R, K, N,
                             _ptr(ws), ws_len, _stream(stream))
    _raise(st, "sd_linear")
    return out


def sd_semi_ar_layer_workspace_size(B, r, d, hq, hkv, I, Lmax):
    return library().sd_semi_ar_layer_workspace_size(B, r, d, hq, hkv, I, Lmax)


SEMI_AR_WEIGHTS = ("fc_w", "fc_b", "ln1", "wqkv", "wo", "ln2", "wgu", "wdown")


def sd_semi_ar_layer(u, weights, k_cache, v_cache, pos, hq, hkv, eps, theta, out=None,
                     workspace=None, stream=None):
    """One draft step of the semi-autoregressive layer.  u [B, r, 2d] bf16;
    weights: dict of fc_w [d, 2d], wqkv [(hq + 2 hkv) D, d], wo [d, hq D],
    wgu [2I, d], wdown [d, I] (bf16) and fc_b, ln1, ln2 [d] (fp32); caches
    [B, Lmax, hkv, D] bf16 (updated in place at positions pos[b] ..
    pos[b] + r - 1); pos [B] int32.  Returns out [B, r, d] fp32."""
    torch = _torch()
    _check(u, "u", dtype=torch.bfloat16, ndim=3)
    B, r, d2 = u.shape
    d = d2 // 2
    for name in SEMI_AR_WEIGHTS:
        t = weights[name]
        _check(t, name, dtype=torch.float32 if name in ("fc_b", "ln1", "ln2") else torch.bfloat16)
    _check(k_cache, "k_cache", dtype=torch.bfloat16, ndim=4)
    _check(v_cache, "v_cache", dtype=torch.bfloat16, ndim=4)
    _check(pos, "pos", dtype=torch.int32, ndim=1)
    Lmax = k_cache.shape[1]
    I = weights["wdown"].shape[1]
    D = d // hq
    shapes = {"fc_w": (d, 2 * d), "fc_b": (d,), "ln1": (d,), "wqkv": ((hq + 2 * hkv) * D, d),
              "wo": (d, hq * D), "ln2": (d,), "wgu": (2 * I, d), "wdown": (d, I)}
    for name, shp in shapes.items():
        if tuple(weights[name].shape) != shp:
            raise ValueError(f"{name} must be {shp}, got {tuple(weights[name].shape)}")
    if tuple(k_cache.shape) != (B, Lmax, hkv, D) or tuple(v_cache.shape) != (B, Lmax, hkv, D):
        raise ValueError("caches must be [B, Lmax, hkv, d / hq]")
    if pos.shape[0] != B:
        raise ValueError("pos must be [B]")
    for name, t in [(n, weights[n]) for n in SEMI_AR_WEIGHTS] + [
            ("k_cache", k_cache), ("v_cache", v_cache), ("pos", pos)]:
        _same_device(name, t, u.device)
    if out is None:
        out = torch.empty((B, r, d), dtype=torch.float32, device=u.device)
    _out(out, "out", (B, r, d), torch.float32, u.device)
    ws_bytes = sd_semi_ar_layer_workspace_size(B, r, d, hq, hkv, I, Lmax)
    ws, ws_len = _workspace(ws_bytes, u.device, workspace)
    W = weights
    st = library().sd_semi_ar_layer(_ptr(u), _ptr(W["fc_w"]), _ptr(W["fc_b"]), _ptr(W["ln1"]),
                                    _ptr(W["wqkv"]), _ptr(W["wo"]), _ptr(W["ln2"]), _ptr(W["wgu"]),
                                    _ptr(W["wdown"]), _ptr(k_cache), _ptr(v_cache), _ptr(pos),
                                    _ptr(out), B, r, d, hq, hkv, I, Lmax, float(eps), float(theta),
                                    _ptr(ws), ws_len, _stream(stream))
    _raise(st, "sd_semi_ar_layer")
    return out


def sd_semi_ar_draft_workspace_size(B, r0, d, hq, hkv, I, Lmax, V, K, kp):
    return library().sd_semi_ar_draft_workspace_size(B, r0, d, hq, hkv, I, Lmax, V, K, kp)


def sd_semi_ar_draft(u0, weights, lm_w, emb, ph, k_cache, v_cache, pos, u, K, kp, hq, hkv, eps, theta,
                     temperature, tokens=None, q=None, workspace=None, stream=None):
    """K drafts in K / kp passes of the semi-AR layer.  u0 [B, r0, 2d] bf16
    (last kp rows placeholders); weights as for sd_semi_ar_layer; lm_w and
    emb [V, d] bf16; ph [2d] bf16; u [B, K] fp32 uniforms.  The caches are
    updated in place.  Returns (tokens [B, K] int32, q [B, K, V] fp32)."""
    torch = _torch()
    _check(u0, "u0", dtype=torch.bfloat16, ndim=3)
    B, r0, d2 = u0.shape
    d = d2 // 2
    _check(lm_w, "lm_w", dtype=torch.bfloat16, ndim=2)
    _check(emb, "emb", dtype=torch.bfloat16, ndim=2)
    _check(ph, "ph", dtype=torch.bfloat16, ndim=1)
    _check(u, "u", dtype=torch.float32, ndim=2)
    V = lm_w.shape[0]
    if lm_w.shape[1] != d or tuple(emb.shape) != (V, d) or ph.shape[0] != 2 * d:
        raise ValueError("lm_w and emb must be [V, d], ph [2d]")
    if tuple(u.shape) != (B, K):
        raise ValueError("u must be [B, K]")
    for name in SEMI_AR_WEIGHTS:
        _check(weights[name], name, dtype=torch.float32 if name in ("fc_b", "ln1", "ln2") else torch.bfloat16)
    _check(k_cache, "k_cache", dtype=torch.bfloat16, ndim=4)
    _check(v_cache, "v_cache", dtype=torch.bfloat16, ndim=4)
    _check(pos, "pos", dtype=torch.int32, ndim=1)
    Lmax = k_cache.shape[1]
    I = weights["wdown"].shape[1]
    D = d // hq
    shapes = {"fc_w": (d, 2 * d), "fc_b": (d,), "ln1": (d,), "wqkv": ((hq + 2 * hkv) * D, d),
              "wo": (d, hq * D), "ln2": (d,), "wgu": (2 * I, d), "wdown": (d, I)}
    for name, shp in shapes.items():
        if tuple(weights[name].shape) != shp:
            raise ValueError(f"{name} must be {shp}, got {tuple(weights[name].shape)}")
    if tuple(k_cache.shape) != (B, Lmax, hkv, D) or tuple(v_cache.shape) != (B, Lmax, hkv, D):
        raise ValueError("caches must be [B, Lmax, hkv, d / hq]")
    if pos.shape[0] != B:
        raise ValueError("pos must be [B]")
    for name, t in [(n, weights[n]) for n in SEMI_AR_WEIGHTS] + [
            ("lm_w", lm_w), ("emb", emb), ("ph", ph), ("k_cache", k_cache),
            ("v_cache", v_cache), ("pos", pos), ("u", u)]:
        _same_device(name, t, u0.device)
    if tokens is None:
        tokens = torch.empty((B, K), dtype=torch.int32, device=u0.device)
    if q is None:
        q = torch.empty((B, K, V), dtype=torch.float32, device=u0.device)
    _out(tokens, "tokens", (B, K), torch.int32, u0.device)
    _out(q, "q", (B, K, V), torch.float32, u0.device)
    ws_bytes = sd_semi_ar_draft_workspace_size(B, r0, d, hq, hkv, I, Lmax, V, K, kp)
    ws, ws_len = _workspace(ws_bytes, u0.device, workspace)
    W = weights
    st = library().sd_semi_ar_draft(_ptr(u0), _ptr(W["fc_w"]), _ptr(W["fc_b"]), _ptr(W["ln1"]),
                                    _ptr(W["wqkv"]), _ptr(W["wo"]), _ptr(W["ln2"]), _ptr(W["wgu"]),
                                    _ptr(W["wdown"]), _ptr(lm_w), _ptr(emb), _ptr(ph), _ptr(k_cache),
                                    _ptr(v_cache), _ptr(pos), _ptr(u), _ptr(tokens), _ptr(q),
                                    B, r0, d, hq, hkv, I, Lmax, V, K, kp, float(eps), float(theta),
                                    float(temperature), _ptr(ws), ws_len, _stream(stream))
    _raise(st, "sd_semi_ar_draft")
    return tokens, q


def sd_linear_q8(x, wq, scale, bias=None, residual=None, out=None, workspace=None, stream=None):
    """y = x (scale * wq)^T (+ bias) (+ residual): x [R, K] bf16, wq [N, K]
    int8, scale [N] fp32.  Returns y [R, N] fp32."""
    torch = _torch()
    _check(x, "x", dtype=torch.bfloat16, ndim=2)
    _check(wq, "wq", dtype=torch.int8, ndim=2)
    _check(scale, "scale", dtype=torch.float32, ndim=1)
    R, K = x.shape
    N = wq.shape[0]
    if wq.shape[1] != K or scale.shape[0] != N:
        raise ValueError("wq must be [N, K] and scale [N]")
    if bias is not None:
        _check(bias, "bias", dtype=torch.float32, ndim=1)
        if bias.shape[0] != N:
            raise ValueError("bias must be [N]")
    if residual is not None:
        _check(residual, "residual", dtype=torch.float32, ndim=2)
        if tuple(residual.shape) != (R, N):
            raise ValueError("residual must be [R, N]")
    for name, t in (("wq", wq), ("scale", scale), ("bias", bias), ("residual", residual)):
        _same_device(name, t, x.device)
    if out is None:
        out = torch.empty((R, N), dtype=torch.float32, device=x.device)
    _out(out, "out", (R, N), torch.float32, x.device)
    ws_bytes = sd_linear_workspace_size(R, K, N)
    ws, ws_len = _workspace(ws_bytes, x.device, workspace)
    st = library().sd_linear_q8(_ptr(x), _ptr(wq), _ptr(scale), _ptr(bias), _ptr(residual), _ptr(out), R, K, N,
                                _ptr(ws), ws_len, _stream(stream))
    _raise(st, "sd_linear_q8")
    return out


Q8_WEIGHTS = ("fc_w", "wqkv", "wo", "wgu", "wdown")


def sd_semi_ar_layer_q8(u, weights, k_cache, v_cache, pos, hq, hkv, eps, theta, out=None, workspace=None,
                        stream=None):
    """sd_semi_ar_layer of the int8 draft: weights holds int8 fc_w, wqkv, wo,
    wgu, wdown and their fp32 row scales under the names + "_s"."""
    torch = _torch()
    _check(u, "u", dtype=torch.bfloat16, ndim=3)
    B, r, d2 = u.shape
    d = d2 // 2
    for name in Q8_WEIGHTS:
        _check(weights[name], name, dtype=torch.int8, ndim=2)
        _check(weights[name + "_s"], name + "_s", dtype=torch.float32, ndim=1)
        if weights[name + "_s"].shape[0] != weights[name].shape[0]:
            raise ValueError(f"{name}_s must hold one scale per row of {name}")
    for name in ("fc_b", "ln1", "ln2"):
        _check(weights[name], name, dtype=torch.float32, ndim=1)
    _check(k_cache, "k_cache", dtype=torch.bfloat16, ndim=4)
    _check(v_cache, "v_cache", dtype=torch.bfloat16, ndim=4)
    _check(pos, "pos", dtype=torch.int32, ndim=1)
    Lmax = k_cache.shape[1]
    I = weights["wdown"].shape[1]
    D = d // hq
    shapes = {"fc_w": (d, 2 * d), "wqkv": ((hq + 2 * hkv) * D, d), "wo": (d, hq * D), "wgu": (2 * I, d),
              "wdown": (d, I)}
    for name, shp in shapes.items():
        if tuple(weights[name].shape) != shp:
            raise ValueError(f"{name} must be {shp}, got {tuple(weights[name].shape)}")
    for name in ("fc_b", "ln1", "ln2"):
        if tuple(weights[name].shape) != (d,):
            raise ValueError(f"{name} must be ({d},)")
    if tuple(k_cache.shape) != (B, Lmax, hkv, D) or tuple(v_cache.shape) != (B, Lmax, hkv, D):
        raise ValueError("caches must be [B, Lmax, hkv, d / hq]")
    if pos.shape[0] != B:
        raise ValueError("pos must be [B]")
    for name, t in [(n, weights[n]) for n in Q8_WEIGHTS] + [
            (n + "_s", weights[n + "_s"]) for n in Q8_WEIGHTS] + [
            (n, weights[n]) for n in ("fc_b", "ln1", "ln2")] + [
            ("k_cache", k_cache), ("v_cache", v_cache), ("pos", pos)]:
        _same_device(name, t, u.device)
    if out is None:
        out = torch.empty((B, r, d), dtype=torch.float32, device=u.device)
    _out(out, "out", (B, r, d), torch.float32, u.device)
    ws_bytes = sd_semi_ar_layer_workspace_size(B, r, d, hq, hkv, I, Lmax)
    ws, ws_len = _workspace(ws_bytes, u.device, workspace)
    W = weights
    st = library().sd_semi_ar_layer_q8(_ptr(u), _ptr(W["fc_w"]), _ptr(W["fc_w_s"]), _ptr(W["fc_b"]),
                                       _ptr(W["ln1"]), _ptr(W["wqkv"]), _ptr(W["wqkv_s"]), _ptr(W["wo"]),
                                       _ptr(W["wo_s"]), _ptr(W["ln2"]), _ptr(W["wgu"]), _ptr(W["wgu_s"]),
                                       _ptr(W["wdown"]), _ptr(W["wdown_s"]), _ptr(k_cache), _ptr(v_cache),
                                       _ptr(pos), _ptr(out), B, r, d, hq, hkv, I, Lmax, float(eps),
                                       float(theta), _ptr(ws), ws_len, _stream(stream))
    _raise(st, "sd_semi_ar_layer_q8")
    return out


def sd_avg_pool_compress(feats, C, out=None, stream=None):
    """Average pooling of feats [B, N, d] (bf16 or fp32) into C contiguous
    token groups.  Returns out [B, C, d] fp32."""
    torch = _torch()
    _check(feats, "feats", ndim=3)
    B, N, d = feats.shape
    if out is None:
        out = torch.empty((B, C, d), dtype=torch.float32, device=feats.device)
    _out(out, "out", (B, C, d), torch.float32, feats.device)
    st = library().sd_avg_pool_compress(_ptr(feats), _ptr(out), B, N, C, d, _dtype_code(feats), _stream(stream))
    _raise(st, "sd_avg_pool_compress")
    return out
