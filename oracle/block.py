"""Float64 oracle of the window-attention block around PnP-Nystra.

Test infrastructure only (see the package header).  The block is the
structure Sec. 1 describes for SwinIR / Uformer-style models: the feature
map is cut into non-overlapping w x w windows (optionally after a cyclic
shift of w // 2 or any s < w, the shifted windows of those models), each
window's tokens are projected to queries, keys and values (Q, K, V = X W),
every head attends independently (d = h d_h), the heads are concatenated and
projected, and the windows are put back in place.  The attention itself is
the PnP-Nystra oracle (Algorithm 1, Eq. (8)) or exact softmax attention
(Eq. (1)).

Relative-position bias and the shifted-window attention mask are not part of
Eqs. (1)-(8); the block has neither (a reading, stated with the others).

Layouts: x and y are [B][H][W][C] (channels last); w_qkv is [C][3C] with
y = x w_qkv (columns: Q, then K, then V; head j of each takes columns
j d_h .. (j+1) d_h - 1); w_proj is [C][C].
"""
import numpy as np

from . import reference


def window_tokens_loops(B, H, W, w, shift):
    """Pixel index (b H + y) W + x of every (window, token), by explicit loops.

    Windows are numbered b-major, then row-major over the (H/w) x (W/w)
    window grid; tokens row-major inside a window.  With a shift s, window
    token (ty, tx) of window (wy, wx) is the pixel ((wy w + ty + s) mod H,
    (wx w + tx + s) mod W): the map rolled by -s before partitioning."""
    nwy, nwx = H // w, W // w
    out = np.empty((B * nwy * nwx, w * w), dtype=np.int64)
    win = 0
    for b in range(B):
        for wy in range(nwy):
            for wx in range(nwx):
                t = 0
                for ty in range(w):
                    for tx in range(w):
                        y = (wy * w + ty + shift) % H
                        x = (wx * w + tx + shift) % W
                        out[win, t] = (b * H + y) * W + x
                        t += 1
                win += 1
    return out


def window_tokens_roll(B, H, W, w, shift):
    """The same index table as array operations: roll, then reshape into
    windows (a second, independent formulation)."""
    idx = np.arange(B * H * W, dtype=np.int64).reshape(B, H, W)
    idx = np.roll(idx, shift=(-shift, -shift), axis=(1, 2))
    idx = idx.reshape(B, H // w, w, W // w, w).transpose(0, 1, 3, 2, 4)
    return idx.reshape(-1, w * w)


def round_bf16(x):
    """Round float64 values to bfloat16 (to float32 first, then the upper 16
    bits, ties to even), returned as float64."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def block_forward(x, w_qkv, b_qkv, w_proj, b_proj, heads, window, shift=0, m=16, iters=6,
                  mode=0, attention="nystrom", dtype="f32", scale=None, n_threads=0,
                  round_output=True):
    """y = block(x).  For dtype "bf16" every tensor the block stores (Q, K,
    V, the attention output, y) is rounded to bf16, as a bf16 model stores
    them; arithmetic is float64 throughout.  round_output=False leaves y
    itself unrounded (the float64 value a bf16 store of y would round), so
    that a comparison can tell y's own rounding from everything before it."""
    x = np.asarray(x, dtype=np.float64)
    B, H, W, C = x.shape
    d = C // heads
    N = window * window
    store = round_bf16 if dtype == "bf16" else (lambda a: a)
    idx = window_tokens_loops(B, H, W, window, shift)          # [nW, N]
    nW = idx.shape[0]
    xw = x.reshape(-1, C)[idx]                                 # [nW, N, C]
    qkv = store(xw @ np.asarray(w_qkv, np.float64) + np.asarray(b_qkv, np.float64))
    qkv = qkv.reshape(nW, N, 3, heads, d).transpose(2, 0, 3, 1, 4)   # [3, nW, heads, N, d]
    q, k, v = (np.ascontiguousarray(qkv[i]) for i in range(3))
    if attention == "nystrom":
        o = reference.forward(q, k, v, m, iters=iters, mode=mode, scale=scale,
                              n_threads=n_threads)
    elif attention == "exact":
        o = reference.exact(q, k, v, scale=scale, n_threads=n_threads)
    else:
        raise ValueError(attention)
    o = store(o)
    ocat = o.transpose(0, 2, 1, 3).reshape(nW, N, C)           # heads concatenated
    yw = ocat @ np.asarray(w_proj, np.float64) + np.asarray(b_proj, np.float64)
    y = np.empty((B * H * W, C))
    y[idx.reshape(-1)] = yw.reshape(-1, C)                     # windows back in place
    y = y.reshape(B, H, W, C)
    return store(y) if round_output else y
