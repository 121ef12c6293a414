"""Thin Python binding of liblla.so (argument marshalling only).

Every entry point forwards torch tensors' device pointers and the current HIP
stream to the C ABI declared in include/lla.h; all computation happens in the
library's HIP kernels.  Torch provides device memory and streams only.

Latent caches are torch tensors of shape [B, H, n_max // 64, r, 64] -- the
paged, feature-major layout the kernels use (logical c[b][h][n][j] is
element [b, h, n // 64, j, n % 64]).  ``to_paged`` / ``from_paged`` convert
between that layout and a token-major [B, H, N, r] tensor (pure views and
copies, no arithmetic).
"""

from __future__ import annotations

import ctypes
import math
import os
from fractions import Fraction

import torch

PAGE = 64
MAX_RANK = 512
MAX_SPLITS = 64

LLA_OK, LLA_ERR_INVALID_ARG, LLA_ERR_UNSUPPORTED, LLA_ERR_WORKSPACE, LLA_ERR_HIP, LLA_ERR_SCRATCH = range(6)
LLA_F32, LLA_BF16 = 0, 1

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblla.so")
ABI_VERSION = 10  # LLA_ABI_VERSION of include/lla.h this binding follows

_c_int, _c_i64, _c_vp, _c_f, _c_sz = (ctypes.c_int, ctypes.c_int64, ctypes.c_void_p,
                                      ctypes.c_float, ctypes.c_size_t)

_SIGS = {
    "lla_status_string": (ctypes.c_char_p, [_c_int]),
    "lla_abi_version": (_c_int, []),
    "lla_rho": (_c_int, [_c_i64] * 4 + [ctypes.POINTER(_c_i64)] * 2),
    "lla_cache_bytes": (_c_int, [_c_i64] * 8 + [_c_int, ctypes.POINTER(_c_i64)]),
    "lla_encode": (_c_int, [_c_int] * 8 + [_c_vp] * 8 + [_c_int, _c_int, _c_vp]),
    "lla_decode_workspace_bytes": (_c_int, [_c_int] * 4 + [ctypes.POINTER(_c_sz)]),
    "lla_decode_splits": (_c_int, [_c_int] * 8 + [ctypes.POINTER(_c_int)]),
    "lla_decode_attn": (_c_int, [_c_int] * 9 + [_c_vp] * 8 + [_c_f, _c_vp, _c_vp, _c_sz, _c_vp]),
    "lla_decode_attn_noalloc": (_c_int, [_c_int] * 9 + [_c_vp] * 8 + [_c_f, _c_vp, _c_vp]),
    "lla_prefill_attn": (_c_int, [_c_int] * 10 + [_c_vp] * 7 + [_c_f, _c_vp, _c_vp, _c_sz, _c_vp]),
    "lla_prefill_workspace_bytes": (_c_int, [_c_int] * 8 + [ctypes.POINTER(_c_sz)]),
    "lla_rope_write": (_c_int, [_c_int] * 5 + [_c_vp, ctypes.c_double, _c_vp, _c_int, _c_int, _c_vp]),
    "lla_rope_rotate": (_c_int, [_c_int] * 5 + [_c_vp, _c_vp, _c_int, ctypes.c_double, _c_vp, _c_vp]),
    "lla_decode_attn_rope": (_c_int, [_c_int] * 11 + [_c_vp] * 10 + [_c_f, _c_vp, _c_vp, _c_sz, _c_vp]),
    "lla_prefill_attn_rope": (_c_int, [_c_int] * 12 + [_c_vp] * 9 + [_c_f, _c_vp, _c_vp]),
    "lla_encode_ring": (_c_int, [_c_int] * 8 + [_c_vp] * 8 + [_c_int] * 4 + [_c_vp]),
    "lla_rope_write_ring": (_c_int, [_c_int] * 5 + [_c_vp, ctypes.c_double, _c_vp] + [_c_int] * 4 + [_c_vp]),
    "lla_encode_2d": (_c_int, [_c_int] * 8 + [_c_vp] * 8 + [_c_int, _c_int, _c_vp, _c_sz, _c_vp]),
    "lla_encode_2d_workspace_bytes": (_c_int, [_c_int] * 7 + [ctypes.POINTER(_c_sz)]),
    "lla_decode_2d_workspace_bytes": (_c_int, [_c_int] * 5 + [ctypes.POINTER(_c_sz)]),
    "lla_decode_attn_2d": (_c_int, [_c_int] * 9 + [_c_vp] * 8 + [_c_f, _c_vp, _c_vp, _c_sz, _c_vp]),
    "lla_prefill_2d_workspace_bytes": (_c_int, [_c_int] * 4 + [ctypes.POINTER(_c_sz)]),
    "lla_prefill_attn_2d": (_c_int, [_c_int] * 10 + [_c_vp] * 7 + [_c_f, _c_vp, _c_vp, _c_sz, _c_vp]),
    "lla_decode_attn_fullrope": (_c_int, [_c_int] * 9 + [_c_vp] * 9 + [ctypes.c_double, _c_f, _c_vp, _c_vp,
                                                                          _c_sz, _c_vp]),
}

_lib = None


def lib() -> ctypes.CDLL:
    """Load liblla.so (built in-tree by paper_2607_15456_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2607_15456_amd.build`")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        if h.lla_abi_version() != ABI_VERSION:  # argument lists differ between versions
            raise RuntimeError(f"{LIB_PATH} has ABI version {h.lla_abi_version()}, this binding "
                               f"needs {ABI_VERSION}; rebuild it")
        _lib = h
    return _lib


class LLAError(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        super().__init__(status_string(status))


def status_string(status: int) -> str:
    return lib().lla_status_string(int(status)).decode()


def _check(status: int) -> None:
    if status != LLA_OK:
        raise LLAError(status)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return LLA_F32
    if t.dtype == torch.bfloat16:
        return LLA_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _out_code(dtype: torch.dtype) -> int:
    return {torch.float32: LLA_F32, torch.bfloat16: LLA_BF16}[dtype]


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(t: torch.Tensor):
    return torch.cuda.current_stream(t.device).cuda_stream


def _need(t: torch.Tensor, name: str, dtype=None, device=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


# ---------------------------------------------------------------------------
# Host-only helpers
# ---------------------------------------------------------------------------

def abi_version() -> int:
    return lib().lla_abi_version()


def rho(T: int, d_head: int, r_k: int, r_v: int) -> Fraction:
    """Exact compression ratio (Sec. 3, Eq. 4) from the library."""
    n, d = _c_i64(), _c_i64()
    _check(lib().lla_rho(T, d_head, r_k, r_v, ctypes.byref(n), ctypes.byref(d)))
    return Fraction(n.value, d.value)


def cache_bytes(layers, heads, T, d_head, r_k, r_v, tokens, elem_bytes, latent) -> int:
    out = _c_i64()
    _check(lib().lla_cache_bytes(layers, heads, T, d_head, r_k, r_v, tokens, elem_bytes,
                                 1 if latent else 0, ctypes.byref(out)))
    return out.value


def decode_workspace_bytes(B: int, H: int, r_v: int, n_ctx: int) -> int:
    out = _c_sz()
    _check(lib().lla_decode_workspace_bytes(B, H, r_v, n_ctx, ctypes.byref(out)))
    return out.value


def decode_splits(dtype: torch.dtype, B: int, H: int, n_ctx: int, r_k: int, r_v: int, d_rope: int = 0,
                  with_workspace: bool = True) -> int:
    """Workgroups lla_decode_attn splits each (b, h) context over (lla_decode_splits)."""
    out = _c_int()
    _check(lib().lla_decode_splits(LLA_BF16 if dtype == torch.bfloat16 else LLA_F32, B, H, n_ctx,
                                   r_k, r_v, d_rope, 1 if with_workspace else 0, ctypes.byref(out)))
    return out.value


# ---------------------------------------------------------------------------
# Cache layout helpers (views and copies only)
# ---------------------------------------------------------------------------

def alloc_cache(B, H, n_max, r, dtype=torch.bfloat16, device="cuda", zero=False):
    if n_max % PAGE:
        raise ValueError("n_max must be a multiple of 64")
    shape = (B, H, n_max // PAGE, r, PAGE)
    return torch.zeros(shape, dtype=dtype, device=device) if zero else torch.empty(shape, dtype=dtype, device=device)


def to_paged(c: torch.Tensor, n_max: int) -> torch.Tensor:
    """[B, H, N, r] token-major -> [B, H, n_max/64, r, 64] paged (positions >= N are zero)."""
    B, H, N, r = c.shape
    if n_max % PAGE or N > n_max:
        raise ValueError("n_max must be a multiple of 64 and >= N")
    full = c.new_zeros((B, H, n_max, r))
    full[:, :, :N] = c
    return full.view(B, H, n_max // PAGE, PAGE, r).transpose(-1, -2).contiguous()


def from_paged(pages: torch.Tensor, n: int | None = None) -> torch.Tensor:
    """[B, H, n_max/64, r, 64] paged -> [B, H, n, r] token-major."""
    B, H, P, r, _ = pages.shape
    out = pages.transpose(-1, -2).reshape(B, H, P * PAGE, r)
    return out if n is None else out[:, :, :n]


def new_workspace(B: int, H: int, r_v: int, n_ctx: int, device="cuda") -> torch.Tensor:
    """A zeroed decode workspace (its arrival counters must start at zero)."""
    return torch.zeros(decode_workspace_bytes(B, H, r_v, n_ctx), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------------------
# Device entry points
# ---------------------------------------------------------------------------

def ring_slot(p: int, sink: int, window: int) -> int:
    """Slot of position p in a sink + window eviction cache (as lla_encode_ring)."""
    return p if p < sink else sink + (p - sink) % window


def encode(x_k, x_v, wdt_k, wdt_v, c_k, c_v, *, T: int, pos0: int, mu_k=None, mu_v=None, evict=None):
    """Write (x - mu) W_down for both axes into cache slots [pos0, pos0 + M) (Eq. 2).

    x_k, x_v: [B, M, H, T*d]; wdt_k: [H, r_k, T*d]; wdt_v: [H, r_v, T*d];
    mu_k, mu_v: [H, T*d] or None; c_k, c_v: paged caches [B, H, n_max/64, r, 64].
    evict = (sink, window): positions go to their ring slots (lla_encode_ring).
    """
    dev = x_k.device
    for t, n in ((x_k, "x_k"), (x_v, "x_v"), (wdt_k, "wdt_k"), (wdt_v, "wdt_v"), (c_k, "c_k"), (c_v, "c_v")):
        _need(t, n, x_k.dtype, dev)
    for t, n in ((mu_k, "mu_k"), (mu_v, "mu_v")):
        if t is not None:
            _need(t, n, x_k.dtype, dev)
    B, M, H, K = x_k.shape
    if K % T:
        raise ValueError("last dim of x must be T * d_head")
    r_k, r_v = wdt_k.shape[1], wdt_v.shape[1]
    n_max = c_k.shape[2] * PAGE
    if (x_v.shape != x_k.shape or wdt_k.shape != (H, r_k, K) or wdt_v.shape != (H, r_v, K)
            or c_k.shape != (B, H, n_max // PAGE, r_k, PAGE) or c_v.shape != (B, H, n_max // PAGE, r_v, PAGE)):
        raise ValueError("inconsistent shapes")
    if evict is None:
        _check(lib().lla_encode(_dt(x_k), B, M, H, T, K // T, r_k, r_v, _ptr(x_k), _ptr(x_v), _ptr(mu_k),
                                _ptr(mu_v), _ptr(wdt_k), _ptr(wdt_v), _ptr(c_k), _ptr(c_v), n_max, pos0,
                                _stream(x_k)))
    else:
        sink, window = evict
        _check(lib().lla_encode_ring(_dt(x_k), B, M, H, T, K // T, r_k, r_v, _ptr(x_k), _ptr(x_v), _ptr(mu_k),
                                     _ptr(mu_v), _ptr(wdt_k), _ptr(wdt_v), _ptr(c_k), _ptr(c_v), n_max, pos0,
                                     sink, window, _stream(x_k)))


def decode_attn(q, c_k, c_v, u_k, u_v, *, n_ctx: int, ctx_len=None, mu_k=None, mu_v=None,
                scale: float | None = None, out=None, out_dtype=torch.float32, workspace=None,
                q_rope=None, r_cache=None):
    """Loop-l decode attention of q [B, H, d] over the paged latent cache.

    u_k: [H, d, r_k], u_v: [H, d, r_v] (loop-l up-projections); mu_*: [H, d] or
    None; ctx_len: int32 device tensor [B] or None (all sequences use n_ctx);
    workspace: from new_workspace() or None (no split-K).  With the decoupled
    rotary branch: q_rope [B, H, d_rope] already rotated (rope_rotate) and
    r_cache the paged rotary cache [B, H_rope, n_max/64, d_rope, 64] (rope_write);
    the default scale is then 1/sqrt(d + d_rope).  Returns out [B, H, d].
    """
    dev = q.device
    B, H, d = q.shape
    for t, n in ((q, "q"), (c_k, "c_k"), (c_v, "c_v"), (u_k, "u_k"), (u_v, "u_v")):
        _need(t, n, q.dtype, dev)
    for t, n in ((mu_k, "mu_k"), (mu_v, "mu_v")):
        if t is not None:
            _need(t, n, q.dtype, dev)
    r_k, r_v = u_k.shape[2], u_v.shape[2]
    n_max = c_k.shape[2] * PAGE
    if (c_k.shape != (B, H, n_max // PAGE, r_k, PAGE) or c_v.shape != (B, H, n_max // PAGE, r_v, PAGE)
            or u_k.shape != (H, d, r_k) or u_v.shape != (H, d, r_v)):
        raise ValueError("inconsistent shapes")
    if ctx_len is not None:
        _need(ctx_len, "ctx_len", torch.int32, dev)
        if ctx_len.shape != (B,):
            raise ValueError("ctx_len must have shape [B]")
    if out is None:
        out = torch.empty((B, H, d), dtype=out_dtype, device=dev)
    else:
        _need(out, "out", None, dev)
    if workspace is not None:
        _need(workspace, "workspace", None, dev)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if (q_rope is None) != (r_cache is None):
        raise ValueError("q_rope and r_cache go together")
    if q_rope is None:
        if scale is None:
            scale = 1.0 / math.sqrt(d)
        _check(lib().lla_decode_attn(_dt(q), _out_code(out.dtype), B, H, d, r_k, r_v, n_max, n_ctx,
                                     _ptr(ctx_len), _ptr(q), _ptr(c_k), _ptr(c_v), _ptr(u_k), _ptr(u_v),
                                     _ptr(mu_k), _ptr(mu_v), float(scale), _ptr(out), _ptr(workspace),
                                     ws_bytes, _stream(q)))
        return out
    H_rope, d_rope = _rope_shapes(q_rope, r_cache, q.dtype, dev, B, H, n_max)
    if q_rope.shape != (B, H, d_rope):
        raise ValueError("q_rope must have shape [B, H, d_rope]")
    if scale is None:
        scale = 1.0 / math.sqrt(d + d_rope)
    _check(lib().lla_decode_attn_rope(_dt(q), _out_code(out.dtype), B, H, d, r_k, r_v, d_rope, H_rope,
                                      n_max, n_ctx, _ptr(ctx_len), _ptr(q), _ptr(q_rope), _ptr(c_k),
                                      _ptr(c_v), _ptr(r_cache), _ptr(u_k), _ptr(u_v), _ptr(mu_k),
                                      _ptr(mu_v), float(scale), _ptr(out), _ptr(workspace), ws_bytes,
                                      _stream(q)))
    return out


def decode_attn_noalloc(q, c_k, c_v, u_k, u_v, *, n_ctx: int, out, ctx_len=None, mu_k=None, mu_v=None,
                        scale: float | None = None):
    """lla_decode_attn_noalloc: decode_attn with no workspace (the library's
    static scratch holds the split-K partials).  ``out`` [B, H, d] is
    caller-allocated (f32 or bf16); nothing is allocated here either."""
    dev = q.device
    B, H, d = q.shape
    for t, n in ((q, "q"), (c_k, "c_k"), (c_v, "c_v"), (u_k, "u_k"), (u_v, "u_v")):
        _need(t, n, q.dtype, dev)
    for t, n in ((mu_k, "mu_k"), (mu_v, "mu_v")):
        if t is not None:
            _need(t, n, q.dtype, dev)
    r_k, r_v = u_k.shape[2], u_v.shape[2]
    n_max = c_k.shape[2] * PAGE
    if (c_k.shape != (B, H, n_max // PAGE, r_k, PAGE) or c_v.shape != (B, H, n_max // PAGE, r_v, PAGE)
            or u_k.shape != (H, d, r_k) or u_v.shape != (H, d, r_v) or out.shape != (B, H, d)):
        raise ValueError("inconsistent shapes")
    _need(out, "out", None, dev)
    if ctx_len is not None:
        _need(ctx_len, "ctx_len", torch.int32, dev)
        if ctx_len.shape != (B,):
            raise ValueError("ctx_len must have shape [B]")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _check(lib().lla_decode_attn_noalloc(_dt(q), _out_code(out.dtype), B, H, d, r_k, r_v, n_max, n_ctx,
                                         _ptr(ctx_len), _ptr(q), _ptr(c_k), _ptr(c_v), _ptr(u_k), _ptr(u_v),
                                         _ptr(mu_k), _ptr(mu_v), float(scale), _ptr(out), _stream(q)))
    return out


def _rope_shapes(q_rope, r_cache, dtype, dev, B, H, n_max):
    _need(q_rope, "q_rope", dtype, dev)
    _need(r_cache, "r_cache", dtype, dev)
    if r_cache.dim() != 5 or r_cache.shape[0] != B or r_cache.shape[2] * PAGE != n_max or r_cache.shape[4] != PAGE:
        raise ValueError("r_cache must be [B, H_rope, n_max/64, d_rope, 64] with the latents' n_max")
    H_rope, d_rope = r_cache.shape[1], r_cache.shape[3]
    if H_rope not in (1, H):
        raise ValueError("r_cache must hold 1 or H rotary keys per token")
    return H_rope, d_rope


def prefill_workspace_bytes(dtype: torch.dtype, B: int, H: int, M: int, d_head: int, r_k: int, r_v: int,
                            p0: int) -> int:
    """Workspace lla_prefill_attn needs (0: none; bf16 ranks above 95 rebuild K and V)."""
    out = _c_sz()
    _check(lib().lla_prefill_workspace_bytes(LLA_BF16 if dtype == torch.bfloat16 else LLA_F32, B, H, M, d_head,
                                             r_k, r_v, p0, ctypes.byref(out)))
    return out.value


def prefill_attn(q, c_k, c_v, u_k, u_v, *, p0: int, mu_k=None, mu_v=None, scale: float | None = None,
                 out=None, out_dtype=torch.float32, q_rope=None, r_cache=None, workspace=None):
    """Causal loop-l prefill of q [B, H, M, d] at positions p0..p0+M-1 over the paged cache.

    workspace: uint8 device tensor of at least prefill_workspace_bytes(...)
    bytes when that is nonzero (allocated here if None).  With the rotary
    branch: q_rope [B, H, M, d_rope] rotated at p0 + m (rope_rotate with
    pos0=p0) and the rotary cache r_cache (rope_write)."""
    dev = q.device
    B, H, M, d = q.shape
    for t, n in ((q, "q"), (c_k, "c_k"), (c_v, "c_v"), (u_k, "u_k"), (u_v, "u_v")):
        _need(t, n, q.dtype, dev)
    for t, n in ((mu_k, "mu_k"), (mu_v, "mu_v")):
        if t is not None:
            _need(t, n, q.dtype, dev)
    r_k, r_v = u_k.shape[2], u_v.shape[2]
    n_max = c_k.shape[2] * PAGE
    if (c_k.shape != (B, H, n_max // PAGE, r_k, PAGE) or c_v.shape != (B, H, n_max // PAGE, r_v, PAGE)
            or u_k.shape != (H, d, r_k) or u_v.shape != (H, d, r_v)):
        raise ValueError("inconsistent shapes")
    if out is None:
        out = torch.empty((B, H, M, d), dtype=out_dtype, device=dev)
    else:
        _need(out, "out", None, dev)
    if (q_rope is None) != (r_cache is None):
        raise ValueError("q_rope and r_cache go together")
    if q_rope is None:
        if scale is None:
            scale = 1.0 / math.sqrt(d)
        if workspace is None:
            need = prefill_workspace_bytes(q.dtype, B, H, M, d, r_k, r_v, p0)
            if need:
                workspace = torch.empty(need, dtype=torch.uint8, device=dev)
        else:
            _need(workspace, "workspace", None, dev)
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        _check(lib().lla_prefill_attn(_dt(q), _out_code(out.dtype), B, H, M, d, r_k, r_v, n_max, p0,
                                      _ptr(q), _ptr(c_k), _ptr(c_v), _ptr(u_k), _ptr(u_v), _ptr(mu_k),
                                      _ptr(mu_v), float(scale), _ptr(out), _ptr(workspace), ws_bytes,
                                      _stream(q)))
        return out
    H_rope, d_rope = _rope_shapes(q_rope, r_cache, q.dtype, dev, B, H, n_max)
    if q_rope.shape != (B, H, M, d_rope):
        raise ValueError("q_rope must have shape [B, H, M, d_rope]")
    if scale is None:
        scale = 1.0 / math.sqrt(d + d_rope)
    _check(lib().lla_prefill_attn_rope(_dt(q), _out_code(out.dtype), B, H, M, d, r_k, r_v, d_rope, H_rope,
                                       n_max, p0, _ptr(q), _ptr(q_rope), _ptr(c_k), _ptr(c_v),
                                       _ptr(r_cache), _ptr(u_k), _ptr(u_v), _ptr(mu_k), _ptr(mu_v),
                                       float(scale), _ptr(out), _stream(q)))
    return out


def rope_write(k_rope, r_cache, *, pos0: int, base: float = 10000.0, evict=None):
    """Rotate the rotary keys k_rope [B, M, H_rope, d_rope] at positions
    pos0..pos0+M-1 and write them into r_cache [B, H_rope, n_max/64, d_rope, 64]
    (into their ring slots when evict = (sink, window))."""
    dev = k_rope.device
    _need(k_rope, "k_rope", None, dev)
    _need(r_cache, "r_cache", k_rope.dtype, dev)
    B, M, G, dr = k_rope.shape
    n_max = r_cache.shape[2] * PAGE
    if r_cache.shape != (B, G, n_max // PAGE, dr, PAGE):
        raise ValueError("inconsistent shapes")
    if evict is None:
        _check(lib().lla_rope_write(_dt(k_rope), B, M, G, dr, _ptr(k_rope), float(base), _ptr(r_cache),
                                    n_max, pos0, _stream(k_rope)))
    else:
        sink, window = evict
        _check(lib().lla_rope_write_ring(_dt(k_rope), B, M, G, dr, _ptr(k_rope), float(base), _ptr(r_cache),
                                         n_max, pos0, sink, window, _stream(k_rope)))


def rope_rotate(x, *, pos=None, pos0: int = 0, base: float = 10000.0, out=None):
    """Rotate rows of x [B, G, M, d_rope] (or [B, G, d_rope], M = 1): row (b, g, m)
    at position (pos[b] if pos is given, else pos0) + m.  pos: int32 device [B]."""
    dev = x.device
    _need(x, "x", None, dev)
    shape = x.shape
    xx = x if x.dim() == 4 else x.unsqueeze(2)
    B, G, M, dr = xx.shape
    if pos is not None:
        _need(pos, "pos", torch.int32, dev)
        if pos.shape != (B,):
            raise ValueError("pos must have shape [B]")
    if out is None:
        out = torch.empty(shape, dtype=x.dtype, device=dev)
    else:
        _need(out, "out", x.dtype, dev)
        if out.shape != shape:
            raise ValueError("out must have x's shape")
    _check(lib().lla_rope_rotate(_dt(x), B, G, M, dr, _ptr(x), _ptr(pos), pos0, float(base), _ptr(out),
                                 _stream(x)))
    return out


# ---------------------------------------------------------------------------
# LLA-2D: one latent per token for all heads
# ---------------------------------------------------------------------------

def alloc_cache_2d(B, n_max, r_k, r_v, dtype=torch.bfloat16, device="cuda"):
    """The LLA-2D caches: keys token-major [B, n_max, r_k], values paged
    feature-major [B, n_max/64, r_v, 64]."""
    if n_max % PAGE:
        raise ValueError("n_max must be a multiple of 64")
    return (torch.empty((B, n_max, r_k), dtype=dtype, device=device),
            torch.empty((B, n_max // PAGE, r_v, PAGE), dtype=dtype, device=device))


def encode_2d_workspace_bytes(B: int, M: int, H: int, T: int, d_head: int, r_k: int, r_v: int) -> int:
    out = _c_sz()
    _check(lib().lla_encode_2d_workspace_bytes(B, M, H, T, d_head, r_k, r_v, ctypes.byref(out)))
    return out.value


def new_encode_2d_workspace(B: int, M: int, H: int, T: int, d_head: int, r_k: int, r_v: int, device="cuda"):
    """A workspace for encode_2d (fp32 partial sums of a split write); None when
    the write takes none."""
    n = encode_2d_workspace_bytes(B, M, H, T, d_head, r_k, r_v)
    return torch.empty(n, dtype=torch.uint8, device=device) if n else None


def encode_2d(x_k, x_v, wdt_k, wdt_v, c_k, c_v, *, T: int, H: int, pos0: int, mu_k=None, mu_v=None,
              workspace=None):
    """LLA-2D write of M new tokens: x_k, x_v [B, M, T*H*d] (loop-major, head-major),
    wdt_* [r, T*H*d], mu_* [T*H*d] or None; caches from alloc_cache_2d.  workspace:
    from new_encode_2d_workspace (splits a decode step's write over the machine)
    or None."""
    dev = x_k.device
    for t, n in ((x_k, "x_k"), (x_v, "x_v"), (wdt_k, "wdt_k"), (wdt_v, "wdt_v"), (c_k, "c_k"), (c_v, "c_v")):
        _need(t, n, x_k.dtype, dev)
    B, M, K = x_k.shape
    if K % (T * H):
        raise ValueError("last dim of x must be T * H * d_head")
    r_k, r_v = wdt_k.shape[0], wdt_v.shape[0]
    n_max = c_k.shape[1]
    if (x_v.shape != x_k.shape or wdt_k.shape != (r_k, K) or wdt_v.shape != (r_v, K)
            or c_k.shape != (B, n_max, r_k) or c_v.shape != (B, n_max // PAGE, r_v, PAGE)):
        raise ValueError("inconsistent shapes")
    _check(lib().lla_encode_2d(_dt(x_k), B, M, H, T, K // (T * H), r_k, r_v, _ptr(x_k), _ptr(x_v), _ptr(mu_k),
                               _ptr(mu_v), _ptr(wdt_k), _ptr(wdt_v), _ptr(c_k), _ptr(c_v), n_max, pos0,
                               _ptr(workspace), 0 if workspace is None else workspace.numel() * workspace.element_size(),
                               _stream(x_k)))


def decode_2d_workspace_bytes(B: int, H: int, r_k: int, r_v: int, n_ctx: int) -> int:
    out = _c_sz()
    _check(lib().lla_decode_2d_workspace_bytes(B, H, r_k, r_v, n_ctx, ctypes.byref(out)))
    return out.value


def decode_attn_2d(q, c_k, c_v, u_k, u_v, *, n_ctx: int, ctx_len=None, mu_k=None, mu_v=None,
                   scale: float | None = None, out=None, out_dtype=torch.float32, workspace=None):
    """LLA-2D loop-l decode of q [B, H, d] over the shared latents (caches from
    alloc_cache_2d); u_k [H, d, r_k], u_v [H, d, r_v].  Returns out [B, H, d]."""
    dev = q.device
    B, H, d = q.shape
    for t, n in ((q, "q"), (c_k, "c_k"), (c_v, "c_v"), (u_k, "u_k"), (u_v, "u_v")):
        _need(t, n, q.dtype, dev)
    r_k, r_v = u_k.shape[2], u_v.shape[2]
    n_max = c_k.shape[1]
    if (c_k.shape != (B, n_max, r_k) or c_v.shape != (B, n_max // PAGE, r_v, PAGE)
            or u_k.shape != (H, d, r_k) or u_v.shape != (H, d, r_v)):
        raise ValueError("inconsistent shapes")
    if ctx_len is not None:
        _need(ctx_len, "ctx_len", torch.int32, dev)
    if out is None:
        out = torch.empty((B, H, d), dtype=out_dtype, device=dev)
    if workspace is None:
        workspace = torch.empty(decode_2d_workspace_bytes(B, H, r_k, r_v, n_ctx), dtype=torch.uint8, device=dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _check(lib().lla_decode_attn_2d(_dt(q), _out_code(out.dtype), B, H, d, r_k, r_v, n_max, n_ctx,
                                    _ptr(ctx_len), _ptr(q), _ptr(c_k), _ptr(c_v), _ptr(u_k), _ptr(u_v),
                                    _ptr(mu_k), _ptr(mu_v), float(scale), _ptr(out), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(), _stream(q)))
    return out


def prefill_2d_workspace_bytes(B: int, H: int, d_head: int, n_keys: int) -> int:
    out = _c_sz()
    _check(lib().lla_prefill_2d_workspace_bytes(B, H, d_head, n_keys, ctypes.byref(out)))
    return out.value


def prefill_attn_2d(q, c_k, c_v, u_k, u_v, *, p0: int = 0, mu_k=None, mu_v=None,
                    scale: float | None = None, out=None, out_dtype=torch.float32, workspace=None):
    """LLA-2D causal prefill of q [B, H, M, d] at positions p0 .. p0+M-1 over the
    shared latents (caches from alloc_cache_2d, filled up to p0+M-1); u_k
    [H, d, r_k], u_v [H, d, r_v].  workspace: uint8 device tensor of at least
    prefill_2d_workspace_bytes(B, H, d, p0 + M) (allocated if None).
    Returns out [B, H, M, d]."""
    dev = q.device
    B, H, M, d = q.shape
    for t, n in ((q, "q"), (c_k, "c_k"), (c_v, "c_v"), (u_k, "u_k"), (u_v, "u_v")):
        _need(t, n, q.dtype, dev)
    r_k, r_v = u_k.shape[2], u_v.shape[2]
    n_max = c_k.shape[1]
    if (c_k.shape != (B, n_max, r_k) or c_v.shape != (B, n_max // PAGE, r_v, PAGE)
            or u_k.shape != (H, d, r_k) or u_v.shape != (H, d, r_v)):
        raise ValueError("inconsistent shapes")
    if out is None:
        out = torch.empty((B, H, M, d), dtype=out_dtype, device=dev)
    if workspace is None:
        workspace = torch.empty(prefill_2d_workspace_bytes(B, H, d, p0 + M), dtype=torch.uint8, device=dev)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _check(lib().lla_prefill_attn_2d(_dt(q), _out_code(out.dtype), B, H, M, d, r_k, r_v, n_max, p0,
                                     _ptr(q), _ptr(c_k), _ptr(c_v), _ptr(u_k), _ptr(u_v), _ptr(mu_k),
                                     _ptr(mu_v), float(scale), _ptr(out), _ptr(workspace),
                                     workspace.numel() * workspace.element_size(), _stream(q)))
    return out


def decode_attn_fullrope(q, c_k, c_v, u_k, u_v, *, n_ctx: int, ctx_len=None, q_pos=None, mu_k=None,
                         mu_v=None, base: float = 10000.0, scale: float | None = None, out=None,
                         out_dtype=torch.float32, workspace=None):
    """Loop-l decode with full RoPE (reconstruct-then-attend) of q [B, H, d]
    (unrotated) over the paged latent cache: keys are rebuilt with U_k and
    rotated at their slot positions, the query at q_pos (int32 device tensor
    [B]; None means each sequence's newest cached token, N_b - 1).  Other
    arguments as decode_attn; the default scale is 1/sqrt(d).  Returns out [B, H, d]."""
    dev = q.device
    B, H, d = q.shape
    for t, n in ((q, "q"), (c_k, "c_k"), (c_v, "c_v"), (u_k, "u_k"), (u_v, "u_v")):
        _need(t, n, q.dtype, dev)
    for t, n in ((mu_k, "mu_k"), (mu_v, "mu_v")):
        if t is not None:
            _need(t, n, q.dtype, dev)
    r_k, r_v = u_k.shape[2], u_v.shape[2]
    n_max = c_k.shape[2] * PAGE
    if (c_k.shape != (B, H, n_max // PAGE, r_k, PAGE) or c_v.shape != (B, H, n_max // PAGE, r_v, PAGE)
            or u_k.shape != (H, d, r_k) or u_v.shape != (H, d, r_v)):
        raise ValueError("inconsistent shapes")
    for t, n in ((ctx_len, "ctx_len"), (q_pos, "q_pos")):
        if t is not None:
            _need(t, n, torch.int32, dev)
            if t.shape != (B,):
                raise ValueError(f"{n} must have shape [B]")
    if out is None:
        out = torch.empty((B, H, d), dtype=out_dtype, device=dev)
    else:
        _need(out, "out", None, dev)
    if workspace is not None:
        _need(workspace, "workspace", None, dev)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _check(lib().lla_decode_attn_fullrope(_dt(q), _out_code(out.dtype), B, H, d, r_k, r_v, n_max, n_ctx,
                                          _ptr(ctx_len), _ptr(q_pos), _ptr(q), _ptr(c_k), _ptr(c_v), _ptr(u_k),
                                          _ptr(u_v), _ptr(mu_k), _ptr(mu_v), float(base), float(scale),
                                          _ptr(out), _ptr(workspace), ws_bytes, _stream(q)))
    return out
