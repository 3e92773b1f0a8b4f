"""ctypes binding of libnystra (include/nystra.h): argument marshalling only.

Every function keeps the name of the C entry point it wraps and forwards
device pointers of torch tensors plus torch's current HIP stream.  No step of
the attention is computed here, and there is no fallback: if libnystra.so is
missing or a call fails, a NystraError is raised.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnystra.so")

F32, BF16 = 0, 1
LM_POOL2D, LM_SEGMENT1D = 0, 1
VARIANT_AUTO, VARIANT_GENERIC, VARIANT_TILED, VARIANT_SPLIT = 0, 1, 2, 3

# Every symbol the header declares.
EXPORTS = (
    "nystra_default_opts", "nystra_attn_forward", "nystra_attn_forward_ex",
    "nystra_exact_attn_forward", "nystra_landmark_pool", "nystra_landmark_map",
    "nystra_select_variant", "nystra_attn_workspace_size", "nystra_attn_forward_ws",
    "nystra_block_workspace_size", "nystra_block_forward", "nystra_attn_forward_noalloc",
    "nystra_block_packed_size", "nystra_block_pack_weights", "nystra_block_forward_packed",
    "nystra_status_str", "nystra_last_error",
)
STATIC_SCRATCH_BYTES = 32 << 20   # NYSTRA_STATIC_SCRATCH_BYTES
BLOCK_NYSTROM, BLOCK_EXACT = 0, 1


class NystraError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        detail = ""
        if _lib is not None:
            detail = _lib.nystra_status_str(status).decode()
            if status == 7:
                detail += ": " + _lib.nystra_last_error().decode()
        super().__init__(f"{where} failed with status {status} ({detail})")


class BlockShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("batch", "height", "width", "channels", "heads",
                                              "window", "shift")]


class Opts(ctypes.Structure):
    _fields_ = [("pinv_iters", ctypes.c_int), ("landmark_mode", ctypes.c_int),
                ("scale", ctypes.c_float), ("variant", ctypes.c_int)]


_lib = None
_vp = ctypes.c_void_p
_i = ctypes.c_int


def lib():
    """The loaded libnystra.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() or "
                          "python paper_2506_08520_amd/build.py")
    L = ctypes.CDLL(LIB_PATH)
    L.nystra_default_opts.argtypes = [ctypes.POINTER(Opts)]
    L.nystra_attn_forward.argtypes = [_vp] * 4 + [_i] * 6 + [_vp]
    L.nystra_attn_forward_ex.argtypes = [_vp] * 4 + [_i] * 6 + [ctypes.POINTER(Opts), _vp]
    L.nystra_exact_attn_forward.argtypes = [_vp] * 4 + [_i] * 5 + [ctypes.c_float, _vp]
    L.nystra_landmark_pool.argtypes = [_vp] * 5 + [_i] * 7 + [_vp]
    L.nystra_landmark_map.argtypes = [_i, _i, _i, _vp]
    L.nystra_select_variant.argtypes = [_i, _i, _i, _i, ctypes.POINTER(Opts)]
    L.nystra_attn_workspace_size.argtypes = [_i] * 6 + [ctypes.POINTER(Opts),
                                                         ctypes.POINTER(ctypes.c_size_t)]
    L.nystra_attn_forward_ws.argtypes = ([_vp] * 4 + [_i] * 6 +
                                         [ctypes.POINTER(Opts), _vp, ctypes.c_size_t, _vp])
    L.nystra_status_str.argtypes = [_i]
    L.nystra_status_str.restype = ctypes.c_char_p
    L.nystra_last_error.argtypes = []
    L.nystra_last_error.restype = ctypes.c_char_p
    L.nystra_block_workspace_size.argtypes = [ctypes.POINTER(BlockShape), _i, _i,
                                              ctypes.POINTER(Opts), _i,
                                              ctypes.POINTER(ctypes.c_size_t)]
    L.nystra_block_forward.argtypes = ([_vp] * 6 + [ctypes.POINTER(BlockShape), _i, _i,
                                                     ctypes.POINTER(Opts), _i, _vp,
                                                     ctypes.c_size_t, _vp])
    L.nystra_attn_forward_noalloc.argtypes = ([_vp] * 4 + [_i] * 6 +
                                              [ctypes.POINTER(Opts), _vp])
    L.nystra_block_packed_size.argtypes = [_i, _i, ctypes.POINTER(ctypes.c_size_t)]
    L.nystra_block_pack_weights.argtypes = [_vp, _vp, _i, _i, _vp, ctypes.c_size_t, _vp]
    L.nystra_block_forward_packed.argtypes = ([_vp] * 6 + [ctypes.c_size_t, _vp,
                                                           ctypes.POINTER(BlockShape), _i, _i,
                                                           ctypes.POINTER(Opts), _i, _vp,
                                                           ctypes.c_size_t, _vp])
    for name in EXPORTS:
        if name not in ("nystra_status_str", "nystra_last_error"):
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(rc, where):
    if rc != 0:
        raise NystraError(rc, where)


def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _shape(q, k, v):
    if q.dim() != 4:
        raise ValueError("tensors must be [n_windows, heads, N, d_h]")
    for t in (q, k, v):
        if t.shape != q.shape or t.dtype != q.dtype or not t.is_contiguous() or not t.is_cuda:
            raise ValueError("Q, K, V must be contiguous device tensors of one shape and dtype")
    return tuple(int(x) for x in q.shape)


def nystra_default_opts():
    o = Opts()
    _check(lib().nystra_default_opts(ctypes.byref(o)), "nystra_default_opts")
    return o


def make_opts(pinv_iters=6, landmark_mode=LM_POOL2D, scale=0.0, variant=VARIANT_AUTO):
    return Opts(pinv_iters, landmark_mode, scale, variant)


def nystra_attn_forward(q, k, v, m, out=None, stream=None):
    """PnP-Nystra with default options; returns O (same shape/dtype as q)."""
    import torch
    W, H, N, d = _shape(q, k, v)
    o = torch.empty_like(q) if out is None else out
    rc = lib().nystra_attn_forward(_ptr(q), _ptr(k), _ptr(v), _ptr(o), W, H, N, d, m,
                                   _dtype_code(q), _stream(stream))
    _check(rc, "nystra_attn_forward")
    return o


def nystra_attn_forward_ex(q, k, v, m, opts=None, out=None, stream=None):
    import torch
    W, H, N, d = _shape(q, k, v)
    o = torch.empty_like(q) if out is None else out
    po = ctypes.byref(opts) if opts is not None else None
    rc = lib().nystra_attn_forward_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(o), W, H, N, d, m,
                                      _dtype_code(q), po, _stream(stream))
    _check(rc, "nystra_attn_forward_ex")
    return o


def nystra_attn_workspace_size(n_windows, heads, N, d_h, m, dtype=F32, opts=None):
    """Bytes of device workspace nystra_attn_forward_ws needs (0: none)."""
    n = ctypes.c_size_t(0)
    po = ctypes.byref(opts) if opts is not None else None
    _check(lib().nystra_attn_workspace_size(n_windows, heads, N, d_h, m, dtype, po,
                                            ctypes.byref(n)), "nystra_attn_workspace_size")
    return int(n.value)


def nystra_attn_forward_ws(q, k, v, m, opts=None, workspace=None, out=None, stream=None):
    """PnP-Nystra through the workspace entry point.  `workspace` is a device
    tensor of at least nystra_attn_workspace_size() bytes; when None, one of
    exactly that size is allocated from torch's allocator (256-byte aligned)."""
    import torch
    W, H, N, d = _shape(q, k, v)
    code = _dtype_code(q)
    o = torch.empty_like(q) if out is None else out
    need = nystra_attn_workspace_size(W, H, N, d, m, code, opts)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    po = ctypes.byref(opts) if opts is not None else None
    rc = lib().nystra_attn_forward_ws(_ptr(q), _ptr(k), _ptr(v), _ptr(o), W, H, N, d, m, code,
                                      po, _ptr(workspace), nbytes, _stream(stream))
    _check(rc, "nystra_attn_forward_ws")
    return o


def nystra_attn_forward_noalloc(q, k, v, m, opts=None, out=None, stream=None):
    """PnP-Nystra through the allocation-free entry point (the token-split
    workspace is the library's static device array)."""
    import torch
    W, H, N, d = _shape(q, k, v)
    o = torch.empty_like(q) if out is None else out
    po = ctypes.byref(opts) if opts is not None else None
    rc = lib().nystra_attn_forward_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), W, H, N, d, m,
                                           _dtype_code(q), po, _stream(stream))
    _check(rc, "nystra_attn_forward_noalloc")
    return o


def nystra_block_workspace_size(shape, m, dtype=F32, opts=None, attention=BLOCK_NYSTROM):
    n = ctypes.c_size_t(0)
    po = ctypes.byref(opts) if opts is not None else None
    _check(lib().nystra_block_workspace_size(ctypes.byref(shape), m, dtype, po, attention,
                                             ctypes.byref(n)), "nystra_block_workspace_size")
    return int(n.value)


def nystra_block_forward(x, w_qkv, b_qkv, w_proj, b_proj, heads, window, shift=0, m=16,
                         opts=None, attention=BLOCK_NYSTROM, workspace=None, out=None,
                         stream=None, packed=None):
    """Window-attention block on x [B, H, W, C] (device, contiguous); returns Y
    of the same shape.  Biases may be None.  The workspace is allocated from
    torch's allocator when not given.  ``packed``: the image from
    nystra_block_pack_weights of these weights (the per-call packing is then
    skipped)."""
    import torch
    if x.dim() != 4 or not x.is_contiguous() or not x.is_cuda:
        raise ValueError("x must be a contiguous device tensor [B, H, W, C]")
    for t in (w_qkv, b_qkv, w_proj, b_proj):
        if t is not None and (t.dtype != x.dtype or not t.is_contiguous() or not t.is_cuda):
            raise ValueError("weights must be contiguous device tensors of x's dtype")
    Bn, H, W, C = (int(v) for v in x.shape)
    shape = BlockShape(Bn, H, W, C, heads, window, shift)
    code = _dtype_code(x)
    need = nystra_block_workspace_size(shape, m, code, opts, attention)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    y = torch.empty_like(x) if out is None else out
    po = ctypes.byref(opts) if opts is not None else None
    if packed is None:
        rc = lib().nystra_block_forward(_ptr(x), _ptr(w_qkv), _ptr(b_qkv), _ptr(w_proj),
                                        _ptr(b_proj), _ptr(y), ctypes.byref(shape), m, code, po,
                                        attention, _ptr(workspace), nbytes, _stream(stream))
        _check(rc, "nystra_block_forward")
    else:
        rc = lib().nystra_block_forward_packed(_ptr(x), _ptr(w_qkv), _ptr(b_qkv), _ptr(w_proj),
                                               _ptr(b_proj), _ptr(packed),
                                               packed.numel() * packed.element_size(), _ptr(y),
                                               ctypes.byref(shape), m, code, po, attention,
                                               _ptr(workspace), nbytes, _stream(stream))
        _check(rc, "nystra_block_forward_packed")
    return y


def nystra_block_packed_size(channels, dtype=F32):
    """Bytes of the packed W_qkv and W_proj image (0 for channels > 256)."""
    n = ctypes.c_size_t(0)
    _check(lib().nystra_block_packed_size(int(channels), dtype, ctypes.byref(n)),
           "nystra_block_packed_size")
    return n.value


def nystra_block_pack_weights(w_qkv, w_proj, out=None, stream=None):
    """Packs w_qkv [C, 3C] and w_proj [C, C] (device, contiguous, one dtype)
    for nystra_block_forward(..., packed=); returns the uint8 image (None for
    channels > 256, where the block reads the weights as given)."""
    import torch
    C = int(w_proj.shape[0])
    for t in (w_qkv, w_proj):
        if t.dtype != w_proj.dtype or not t.is_contiguous() or not t.is_cuda:
            raise ValueError("weights must be contiguous device tensors of one dtype")
    if tuple(w_qkv.shape) != (C, 3 * C) or tuple(w_proj.shape) != (C, C):
        raise ValueError("expected w_qkv [C, 3C] and w_proj [C, C]")
    code = _dtype_code(w_proj)
    need = nystra_block_packed_size(C, code)
    if need == 0:
        return None
    if out is None:
        out = torch.empty(need, dtype=torch.uint8, device=w_proj.device)
    rc = lib().nystra_block_pack_weights(_ptr(w_qkv), _ptr(w_proj), C, code, _ptr(out),
                                         out.numel(), _stream(stream))
    _check(rc, "nystra_block_pack_weights")
    return out


def nystra_exact_attn_forward(q, k, v, scale=0.0, out=None, stream=None):
    import torch
    W, H, N, d = _shape(q, k, v)
    o = torch.empty_like(q) if out is None else out
    rc = lib().nystra_exact_attn_forward(_ptr(q), _ptr(k), _ptr(v), _ptr(o), W, H, N, d,
                                         _dtype_code(q), float(scale), _stream(stream))
    _check(rc, "nystra_exact_attn_forward")
    return o


def nystra_landmark_pool(q, k, m, mode=LM_POOL2D, with_map=True, stream=None):
    """Step 1 alone: (Qbar, Kbar) fp32 [W, H, m, d] and the int32[N] map."""
    import torch
    W, H, N, d = _shape(q, k, q)
    qb = torch.empty((W, H, m, d), dtype=torch.float32, device=q.device)
    kb = torch.empty_like(qb)
    mp = torch.empty(N, dtype=torch.int32, device=q.device) if with_map else None
    rc = lib().nystra_landmark_pool(_ptr(q), _ptr(k), _ptr(qb), _ptr(kb), _ptr(mp), W, H, N,
                                    d, m, _dtype_code(q), mode, _stream(stream))
    _check(rc, "nystra_landmark_pool")
    return qb, kb, mp


def nystra_landmark_map(N, m, mode=LM_POOL2D):
    out = np.zeros(N, dtype=np.int32)
    _check(lib().nystra_landmark_map(N, m, mode, out.ctypes.data_as(ctypes.c_void_p)),
           "nystra_landmark_map")
    return out


def nystra_select_variant(N, d_h, m, dtype=F32, opts=None):
    po = ctypes.byref(opts) if opts is not None else None
    r = lib().nystra_select_variant(N, d_h, m, dtype, po)
    if r < 0:
        raise NystraError(-r, "nystra_select_variant")
    return r


def nystra_status_str(status):
    return lib().nystra_status_str(status).decode()
