"""Python binding of libism_attn.so (ctypes; argument marshalling only).

Every function takes torch tensors already on the GPU, allocates the outputs
and the workspace with torch, passes raw pointers and torch's current HIP
stream to the C ABI, and raises on any status other than ISM_OK. There is no
fallback: if the library is not built or no gfx950 device is present, the
call fails loudly.

Names follow the C ABI (include/ism_attn.h): fwd, bwd, visibility,
prefill_cached, prefill_cached_segment, decode, decode_noalloc,
prefill_paged, decode_paged, positions_2d, rope2d_, prefill_cached_rope2d,
plus check_segments_host and workspace_size. Outputs are allocated with
torch unless the caller passes them (``out=``).
"""

from __future__ import annotations

import ctypes
import math
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libism_attn.so")

ISM_OP_FWD, ISM_OP_BWD, ISM_OP_PREFILL_CACHED, ISM_OP_DECODE = range(4)
ISM_DTYPE_BF16, ISM_DTYPE_F32 = range(2)
ROPE_BASE = 10000.0
STATUS = {0: "ISM_OK", 1: "ISM_ERR_NULL", 2: "ISM_ERR_SHAPE",
          3: "ISM_ERR_UNSUPPORTED", 4: "ISM_ERR_SEGMENTS",
          5: "ISM_ERR_WORKSPACE", 6: "ISM_ERR_CAPACITY",
          7: "ISM_ERR_NO_DEVICE", 8: "ISM_ERR_HIP"}


class IsmError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status


class ism_segments(ctypes.Structure):
    _fields_ = [("cu_seqlens", ctypes.c_void_p),
                ("cu_segs", ctypes.c_void_p),
                ("seg_is_query", ctypes.c_void_p),
                ("batch", ctypes.c_int32),
                ("num_segs", ctypes.c_int32),
                ("total_tokens", ctypes.c_int32),
                ("max_seqlen", ctypes.c_int32)]


_P = ctypes.c_void_p
_I = ctypes.c_int32
_F = ctypes.c_float
_Z = ctypes.c_size_t

_SIGS = {
    "ism_attn_workspace_size": (_Z, [_I, _I, _I, _I, _I, _I, _I, _I]),
    "ism_attn_fwd": (_I, [ctypes.POINTER(ism_segments), _P, _P, _P, _P, _P,
                          _I, _I, _I, _F, _P, _Z, _P]),
    "ism_attn_bwd": (_I, [ctypes.POINTER(ism_segments), _P, _P, _P, _P, _P,
                          _P, _P, _P, _P, _I, _I, _I, _F, _I, _P, _Z, _P]),
    "ism_attn_prefill_cached": (_I, [_P, _I, _I, _I, _P, _P, _P, _P, _P, _I,
                                     _P, _P, _P, _I, _I, _I, _F, _P, _Z, _P]),
    "ism_attn_prefill_cached_segment": (_I, [_P, _I, _I, _I, _I, _P, _P, _P,
                                             _P, _P, _I, _P, _P, _P, _I, _I,
                                             _I, _F, _P, _Z, _P]),
    "ism_attn_prefill_paged": (_I, [_P, _I, _I, _I, _I, _P, _P, _P, _P, _P,
                                    _I, _I, _P, _I, _P, _P, _P, _I, _I, _I,
                                    _F, _P, _Z, _P]),
    "ism_attn_decode_paged": (_I, [_P, _P, _P, _P, _P, _I, _I, _P, _I, _P,
                                   _I, _I, _P, _P, _I, _I, _I, _F, _I, _P,
                                   _Z, _P]),
    "ism_attn_decode": (_I, [_P, _P, _P, _P, _P, _I, _P, _I, _I, _P, _P, _I,
                             _I, _I, _F, _I, _P, _Z, _P]),
    "ism_attn_decode_noalloc": (_I, [_P, _P, _P, _P, _P, _I, _P, _I, _I, _P,
                                     _P, _I, _I, _I, _F, _I, _P]),
    "ism_visibility": (_I, [ctypes.POINTER(ism_segments), _P, _P, _P]),
    "ism_positions_2d": (_I, [ctypes.POINTER(ism_segments), _P, _P, _P]),
    "ism_rope2d": (_I, [_P, _I, _I, _I, _I, _P, _P, _F, _I, _P]),
    "ism_attn_prefill_cached_rope2d": (_I, [_P, _I, _I, _I, _I, _P, _P, _P,
                                            _P, _P, _I, _P, _P, _P, _F, _P,
                                            _P, _I, _I, _I, _F, _P, _Z,
                                            _P]),
    "ism_check_segments_host": (_I, [_P, _P, _P, _I, _I, _I, _I]),
    "ism_status_string": (ctypes.c_char_p, [_I]),
    "ism_last_error": (ctypes.c_char_p, []),
    "ism_version": (ctypes.c_char_p, []),
}

_lib = None


def lib():
    """Load the library once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2408_00539_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status):
    if status != 0:
        raise IsmError(status, lib().ism_last_error().decode())


def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _need(t, name, dtype, shape=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU (got {t.device})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {shape}")


def workspace_size(op, batch=0, total_tokens=0, max_seqlen=0, hq=0, hkv=0,
                   d=0, num_splits=0):
    return int(lib().ism_attn_workspace_size(op, batch, total_tokens,
                                             max_seqlen, hq, hkv, d,
                                             num_splits))


def _outputs(out, specs, device):
    """Caller-provided outputs (checked) or new torch tensors.

    specs: one (name, dtype, shape) per output; shape None = absent (the
    caller's entry must then be None too)."""
    torch = _torch()
    if out is None:
        return tuple(None if shp is None else
                     torch.empty(shp, dtype=dt, device=device)
                     for _, dt, shp in specs)
    out = tuple(out)
    if len(out) != len(specs):
        raise ValueError(f"out must hold {len(specs)} tensors")
    for t, (name, dt, shp) in zip(out, specs):
        if shp is None:
            if t is not None:
                raise ValueError(f"{name} is not produced by this call")
            continue
        _need(t, name, dt, shp)
    return out


def _workspace(nbytes, device):
    torch = _torch()
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


class Segments:
    """Device-resident dialogue structure of a packed batch.

    cu_seqlens [B+1] int32, cu_segs [S+1] int32, seg_is_query [S] uint8,
    plus host scalars. ``from_host`` uploads numpy arrays.
    """

    def __init__(self, cu_seqlens, cu_segs, seg_is_query, total_tokens,
                 max_seqlen):
        torch = _torch()
        _need(cu_seqlens, "cu_seqlens", torch.int32)
        _need(cu_segs, "cu_segs", torch.int32)
        _need(seg_is_query, "seg_is_query", torch.uint8)
        self.cu_seqlens, self.cu_segs, self.seg_is_query = (
            cu_seqlens, cu_segs, seg_is_query)
        self.batch = cu_seqlens.numel() - 1
        self.num_segs = seg_is_query.numel()
        self.total_tokens = int(total_tokens)
        self.max_seqlen = int(max_seqlen)

    @classmethod
    def from_host(cls, cu_seqlens, cu_segs, seg_is_query, device="cuda"):
        import numpy as np
        torch = _torch()
        cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
        return cls(torch.from_numpy(cu).to(device),
                   torch.from_numpy(np.ascontiguousarray(cu_segs, np.int32)).to(device),
                   torch.from_numpy(np.ascontiguousarray(seg_is_query, np.uint8)).to(device),
                   int(cu[-1]), int(np.max(np.diff(cu))))

    def c_struct(self):
        return ism_segments(self.cu_seqlens.data_ptr(), self.cu_segs.data_ptr(),
                            self.seg_is_query.data_ptr(), self.batch,
                            self.num_segs, self.total_tokens, self.max_seqlen)


def fwd(q, k, v, segs, scale=None, return_lse=True, out=None):
    """ISM forward over packed dialogues. q [T,hq,d], k/v [T,hkv,d] bf16.
    Returns (o bf16 [T,hq,d], lse fp32 [hq,T] or None); ``out=(o, lse)``
    writes into caller tensors instead."""
    torch = _torch()
    _need(q, "q", torch.bfloat16)
    if q.dim() != 3:
        raise ValueError("q must be [T, hq, d]")
    T, hq, d = q.shape
    hkv = k.shape[1] if k.dim() == 3 else -1
    _need(k, "k", torch.bfloat16, (T, hkv, d))
    _need(v, "v", torch.bfloat16, (T, hkv, d))
    if T != segs.total_tokens:
        raise ValueError("q rows != segs.total_tokens")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    o, lse = _outputs(out, [("o", torch.bfloat16, (T, hq, d)),
                            ("lse", torch.float32,
                             (hq, T) if return_lse else None)], q.device)
    nws = workspace_size(ISM_OP_FWD, segs.batch, T, segs.max_seqlen, hq, hkv, d)
    ws = _workspace(nws, q.device)
    sg = segs.c_struct()
    _check(lib().ism_attn_fwd(ctypes.byref(sg), _ptr(q), _ptr(k), _ptr(v),
                              _ptr(o), _ptr(lse), hq, hkv, d, scale, _ptr(ws),
                              nws, _stream()))
    return o, lse


def bwd(q, k, v, o, lse, dout, segs, scale=None, deterministic=False,
        out=None):
    """Gradients (dq [T,hq,d], dk, dv [T,hkv,d], fp32) of ism fwd;
    ``out=(dq, dk, dv)`` writes into caller tensors instead. The result is
    bitwise repeatable whatever ``deterministic`` says (see ism_attn_bwd)."""
    torch = _torch()
    _need(q, "q", torch.bfloat16)
    if q.dim() != 3:
        raise ValueError("q must be [T, hq, d]")
    T, hq, d = q.shape
    hkv = k.shape[1] if k.dim() == 3 else -1
    _need(k, "k", torch.bfloat16, (T, hkv, d))
    _need(v, "v", torch.bfloat16, (T, hkv, d))
    _need(o, "o", torch.bfloat16, (T, hq, d))
    _need(dout, "dout", torch.bfloat16, (T, hq, d))
    _need(lse, "lse", torch.float32, (hq, T))
    if T != segs.total_tokens:
        raise ValueError("q rows != segs.total_tokens")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dq, dk, dv = _outputs(out, [("dq", torch.float32, (T, hq, d)),
                                ("dk", torch.float32, (T, hkv, d)),
                                ("dv", torch.float32, (T, hkv, d))], q.device)
    nws = workspace_size(ISM_OP_BWD, segs.batch, T, segs.max_seqlen, hq, hkv, d)
    ws = _workspace(nws, q.device)
    sg = segs.c_struct()
    _check(lib().ism_attn_bwd(ctypes.byref(sg), _ptr(q), _ptr(k), _ptr(v),
                              _ptr(o), _ptr(lse), _ptr(dout), _ptr(dq),
                              _ptr(dk), _ptr(dv), hq, hkv, d, scale,
                              1 if deterministic else 0, _ptr(ws), nws,
                              _stream()))
    return dq, dk, dv


def prefill_cached(q_new, k_new, v_new, k_cache, v_cache, cache_seqlens,
                   cu_seqlens_new, max_new, scale=None, return_lse=True,
                   out=None):
    """New query segment against the reused cache (appends k_new/v_new).
    Returns (o [Tn,hq,d] bf16, lse [hq,Tn] fp32 or None). A dialogue whose
    C_b + L_b exceeds the cache gets NaN rows (the library cannot see the
    device lengths before the launch)."""
    return _prefill(None, q_new, k_new, v_new, k_cache, v_cache,
                    cache_seqlens, cu_seqlens_new, max_new, scale, return_lse,
                    out)


def prefill_cached_segment(q_new, k_new, v_new, k_cache, v_cache,
                           cache_seqlens, cu_seqlens_new, max_new,
                           seg_is_query, scale=None, return_lse=True,
                           out=None):
    """New segment against the reused cache: a query segment (every new row
    sees the whole cache and all new rows) or, with seg_is_query false, an
    answer segment (new row r sees the cache and new rows 0..r)."""
    return _prefill(bool(seg_is_query), q_new, k_new, v_new, k_cache,
                    v_cache, cache_seqlens, cu_seqlens_new, max_new, scale,
                    return_lse, out)


def _prefill(seg_is_query, q_new, k_new, v_new, k_cache, v_cache,
             cache_seqlens, cu_seqlens_new, max_new, scale, return_lse,
             out=None):
    torch = _torch()
    Tn, hq, d = q_new.shape
    B, hkv, cap, _ = k_cache.shape
    _need(q_new, "q_new", torch.bfloat16)
    _need(k_new, "k_new", torch.bfloat16, (Tn, hkv, d))
    _need(v_new, "v_new", torch.bfloat16, (Tn, hkv, d))
    _need(k_cache, "k_cache", torch.bfloat16, (B, hkv, cap, d))
    _need(v_cache, "v_cache", torch.bfloat16, (B, hkv, cap, d))
    _need(cache_seqlens, "cache_seqlens", torch.int32, (B,))
    _need(cu_seqlens_new, "cu_seqlens_new", torch.int32, (B + 1,))
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    o, lse = _outputs(out, [("o", torch.bfloat16, (Tn, hq, d)),
                            ("lse", torch.float32,
                             (hq, Tn) if return_lse else None)], q_new.device)
    if seg_is_query is None:
        _check(lib().ism_attn_prefill_cached(
            _ptr(cu_seqlens_new), B, Tn, int(max_new), _ptr(q_new),
            _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), cap,
            _ptr(cache_seqlens), _ptr(o), _ptr(lse), hq, hkv, d, scale, None,
            0, _stream()))
    else:
        _check(lib().ism_attn_prefill_cached_segment(
            _ptr(cu_seqlens_new), B, Tn, int(max_new), int(seg_is_query),
            _ptr(q_new), _ptr(k_new), _ptr(v_new), _ptr(k_cache),
            _ptr(v_cache), cap, _ptr(cache_seqlens), _ptr(o), _ptr(lse), hq,
            hkv, d, scale, None, 0, _stream()))
    return o, lse


def positions_2d(segs):
    """2-D positions (pos1 = segment index in the dialogue, pos2 = offset in
    the segment) of every token of a packed batch: two int32 [T] tensors."""
    torch = _torch()
    dev = segs.cu_seqlens.device
    pos1 = torch.empty(segs.total_tokens, dtype=torch.int32, device=dev)
    pos2 = torch.empty_like(pos1)
    st = segs.c_struct()
    _check(lib().ism_positions_2d(ctypes.byref(st), _ptr(pos1), _ptr(pos2), _stream()))
    return pos1, pos2


def rope2d_(x, pos1, pos2, base=ROPE_BASE, inverse=False):
    """Rotate x [T, heads, d] (bf16 or fp32) in place by the 2-D positions
    pos1, pos2 [T] int32; ``inverse`` rotates back (for gradients)."""
    torch = _torch()
    if x.dim() != 3 or not x.is_contiguous():
        raise ValueError("x must be a contiguous [T, heads, d] tensor")
    if x.dtype == torch.bfloat16:
        dt = ISM_DTYPE_BF16
    elif x.dtype == torch.float32:
        dt = ISM_DTYPE_F32
    else:
        raise ValueError(f"x must be bf16 or fp32, got {x.dtype}")
    T, H, d = x.shape
    _need(pos1, "pos1", torch.int32, (T,))
    _need(pos2, "pos2", torch.int32, (T,))
    _check(lib().ism_rope2d(_ptr(x), dt, T, H, d, _ptr(pos1), _ptr(pos2), float(base),
                            int(bool(inverse)), _stream()))
    return x


def prefill_cached_rope2d(q_new, k_new, v_new, k_cache, v_cache, cache_seqlens,
                          cu_seqlens_new, max_new, pos1_new, pos2_new,
                          seg_is_query=True, base=ROPE_BASE, scale=None,
                          return_lse=True):
    """prefill_cached_segment with the new tokens' 2-D positions: keys are
    rotated into the cache, queries as they are loaded (q_new and k_new
    themselves are left unrotated)."""
    torch = _torch()
    Tn, hq, d = q_new.shape
    B, hkv, cap, _ = k_cache.shape
    _need(q_new, "q_new", torch.bfloat16)
    _need(k_new, "k_new", torch.bfloat16, (Tn, hkv, d))
    _need(v_new, "v_new", torch.bfloat16, (Tn, hkv, d))
    _need(k_cache, "k_cache", torch.bfloat16, (B, hkv, cap, d))
    _need(v_cache, "v_cache", torch.bfloat16, (B, hkv, cap, d))
    _need(cache_seqlens, "cache_seqlens", torch.int32, (B,))
    _need(cu_seqlens_new, "cu_seqlens_new", torch.int32, (B + 1,))
    _need(pos1_new, "pos1_new", torch.int32, (Tn,))
    _need(pos2_new, "pos2_new", torch.int32, (Tn,))
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    o = torch.empty_like(q_new)
    lse = torch.empty((hq, Tn), dtype=torch.float32, device=q_new.device) \
        if return_lse else None
    _check(lib().ism_attn_prefill_cached_rope2d(
        _ptr(cu_seqlens_new), B, Tn, int(max_new), int(bool(seg_is_query)),
        _ptr(q_new), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), cap,
        _ptr(cache_seqlens), _ptr(pos1_new), _ptr(pos2_new), float(base), _ptr(o),
        _ptr(lse), hq, hkv, d, scale, None, 0, _stream()))
    return o, lse


def _decode_args(q, k_new, v_new, k_cache, v_cache, cache_seqlens, scale,
                 return_lse, out):
    torch = _torch()
    _need(q, "q", torch.bfloat16)
    if q.dim() != 3 or k_cache.dim() != 4:
        raise ValueError("q must be [B, hq, d], k_cache [B, hkv, cap, d]")
    B, hq, d = q.shape
    _, hkv, cap, _ = k_cache.shape
    _need(k_new, "k_new", torch.bfloat16, (B, hkv, d))
    _need(v_new, "v_new", torch.bfloat16, (B, hkv, d))
    _need(k_cache, "k_cache", torch.bfloat16, (B, hkv, cap, d))
    _need(v_cache, "v_cache", torch.bfloat16, (B, hkv, cap, d))
    _need(cache_seqlens, "cache_seqlens", torch.int32, (B,))
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    o, lse = _outputs(out, [("o", torch.bfloat16, (B, hq, d)),
                            ("lse", torch.float32,
                             (hq, B) if return_lse else None)], q.device)
    return B, hq, hkv, d, cap, scale, o, lse


def decode(q, k_new, v_new, k_cache, v_cache, cache_seqlens, max_seqlen=0,
           scale=None, num_splits=0, return_lse=True, workspace=None,
           out=None):
    """One decode step (appends k_new/v_new at cache_seqlens[b]).
    Returns (o [B,hq,d] bf16, lse [hq,B] fp32 or None). A dialogue whose
    position lies outside the cache gets NaN (nothing is appended)."""
    B, hq, hkv, d, cap, scale, o, lse = _decode_args(
        q, k_new, v_new, k_cache, v_cache, cache_seqlens, scale, return_lse,
        out)
    ms = cap if not max_seqlen else int(max_seqlen)
    nws = workspace_size(ISM_OP_DECODE, B, 0, ms, hq, hkv, d, num_splits)
    ws = workspace if workspace is not None else _workspace(nws, q.device)
    _check(lib().ism_attn_decode(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), cap,
        _ptr(cache_seqlens), B, ms, _ptr(o), _ptr(lse), hq, hkv, d, scale,
        int(num_splits), _ptr(ws), nws if workspace is None else
        workspace.numel(), _stream()))
    return o, lse


def decode_noalloc(q, k_new, v_new, k_cache, v_cache, cache_seqlens,
                   max_seqlen=0, scale=None, num_splits=0, return_lse=True,
                   out=None):
    """The decode step through ism_attn_decode_noalloc: the library itself
    allocates nothing (split partials in its fixed per-device scratch);
    with ``out=(o, lse)`` this wrapper allocates nothing either."""
    B, hq, hkv, d, cap, scale, o, lse = _decode_args(
        q, k_new, v_new, k_cache, v_cache, cache_seqlens, scale, return_lse,
        out)
    _check(lib().ism_attn_decode_noalloc(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), cap,
        _ptr(cache_seqlens), B, int(max_seqlen), _ptr(o), _ptr(lse), hq, hkv,
        d, scale, int(num_splits), _stream()))
    return o, lse


def visibility(segs):
    """Eq. 5 visibility metadata as the kernels compute it: lim [T] (last
    key each token sees) and seer [T] (first token that sees each key),
    int32 on the GPU."""
    torch = _torch()
    dev = segs.cu_seqlens.device
    lim_ = torch.empty(segs.total_tokens, dtype=torch.int32, device=dev)
    seer = torch.empty_like(lim_)
    st = segs.c_struct()
    _check(lib().ism_visibility(ctypes.byref(st), _ptr(lim_), _ptr(seer),
                                _stream()))
    return lim_, seer


def check_segments_host(cu_seqlens, cu_segs, seg_is_query, max_seqlen=None):
    """Validate host (numpy) segment arrays with the library's checker.
    Returns (status, detail)."""
    import numpy as np
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    cs = np.ascontiguousarray(cu_segs, dtype=np.int32)
    fl = np.ascontiguousarray(seg_is_query, dtype=np.uint8)
    ms = int(np.max(np.diff(cu))) if max_seqlen is None and len(cu) > 1 \
        else int(max_seqlen or 0)
    st = lib().ism_check_segments_host(
        cu.ctypes.data, cs.ctypes.data, fl.ctypes.data, len(cu) - 1, len(fl),
        int(cu[-1]) if len(cu) else 0, ms)
    return st, lib().ism_last_error().decode()


def _need_pages(k_pages, v_pages, block_table, hkv, d):
    torch = _torch()
    P, hk, ps, dd = k_pages.shape
    _need(k_pages, "k_pages", torch.bfloat16, (P, hkv, ps, d))
    _need(v_pages, "v_pages", torch.bfloat16, (P, hkv, ps, d))
    _need(block_table, "block_table", torch.int32)
    if block_table.dim() != 2:
        raise ValueError("block_table must be [batch, max_pages]")
    return P, ps, block_table.shape[1]


def prefill_paged(q_new, k_new, v_new, k_pages, v_pages, block_table,
                  cache_seqlens, cu_seqlens_new, max_new, seg_is_query=True,
                  scale=None, return_lse=True):
    """New segment against a paged cache (appends k_new/v_new into the
    pages block_table names). k_pages/v_pages [P, hkv, page_size, d] bf16,
    block_table [B, max_pages] int32. Returns (o, lse)."""
    torch = _torch()
    Tn, hq, d = q_new.shape
    hkv = k_new.shape[1]
    P, ps, mp = _need_pages(k_pages, v_pages, block_table, hkv, d)
    B = block_table.shape[0]
    _need(q_new, "q_new", torch.bfloat16)
    _need(k_new, "k_new", torch.bfloat16, (Tn, hkv, d))
    _need(v_new, "v_new", torch.bfloat16, (Tn, hkv, d))
    _need(cache_seqlens, "cache_seqlens", torch.int32, (B,))
    _need(cu_seqlens_new, "cu_seqlens_new", torch.int32, (B + 1,))
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    o = torch.empty_like(q_new)
    lse = torch.empty((hq, Tn), dtype=torch.float32, device=q_new.device) \
        if return_lse else None
    _check(lib().ism_attn_prefill_paged(
        _ptr(cu_seqlens_new), B, Tn, int(max_new), int(bool(seg_is_query)),
        _ptr(q_new), _ptr(k_new), _ptr(v_new), _ptr(k_pages), _ptr(v_pages),
        P, ps, _ptr(block_table), mp, _ptr(cache_seqlens), _ptr(o), _ptr(lse),
        hq, hkv, d, scale, None, 0, _stream()))
    return o, lse


def decode_paged(q, k_new, v_new, k_pages, v_pages, block_table,
                 cache_seqlens, max_seqlen=0, scale=None, num_splits=0,
                 return_lse=True, workspace=None):
    """One decode step against a paged cache (appends k_new/v_new at
    cache_seqlens[b]). Returns (o [B,hq,d] bf16, lse [hq,B] fp32 or None)."""
    torch = _torch()
    B, hq, d = q.shape
    hkv = k_new.shape[1]
    P, ps, mp = _need_pages(k_pages, v_pages, block_table, hkv, d)
    _need(q, "q", torch.bfloat16)
    _need(k_new, "k_new", torch.bfloat16, (B, hkv, d))
    _need(v_new, "v_new", torch.bfloat16, (B, hkv, d))
    _need(cache_seqlens, "cache_seqlens", torch.int32, (B,))
    if block_table.shape[0] != B:
        raise ValueError("block_table rows != batch")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    cap = mp * ps
    ms = cap if not max_seqlen else int(max_seqlen)
    nws = workspace_size(ISM_OP_DECODE, B, 0, ms, hq, hkv, d, num_splits)
    ws = workspace if workspace is not None else _workspace(nws, q.device)
    o = torch.empty_like(q)
    lse = torch.empty((hq, B), dtype=torch.float32, device=q.device) \
        if return_lse else None
    _check(lib().ism_attn_decode_paged(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pages), _ptr(v_pages), P, ps,
        _ptr(block_table), mp, _ptr(cache_seqlens), B, int(max_seqlen),
        _ptr(o), _ptr(lse), hq, hkv, d, scale, int(num_splits), _ptr(ws),
        nws if workspace is None else workspace.numel(), _stream()))
    return o, lse
