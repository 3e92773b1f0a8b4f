"""Seeded synthetic inputs for window attention (Q, K, V per window and head).

This module only draws and lays out inputs.  It holds none of the attention
method's arithmetic, so both the HIP path and the float64 oracle can take
their inputs from it.

Every array is produced in float64 and then rounded once to the storage type
(fp32 round-to-nearest, or bf16 round-to-nearest-even from the fp32 value); the
returned float64 arrays hold those rounded values exactly, so the oracle reads
precisely what the GPU reads.

Layout of every tensor: [n_windows][heads][N][d_h].  Windows are taken
row-major over the feature map, tokens row-major inside a sqrt(N) x sqrt(N)
window, and head h owns channels [h*d_h, (h+1)*d_h).

The paper measures pretrained SwinIR / Uformer-B / Dehazeformer on public
image-restoration datasets; neither the weights nor the datasets are used here.
These recipes stand in for them with the shapes of those models' attention
layers (SwinIR: 180 channels, 6 heads, 8x8 windows; Uformer-B stage 1: 32
channels, 1 head; enlarged 16x16 and 32x32 windows as in the paper's
restoration experiments).
"""
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    n_windows: int
    heads: int
    N: int          # tokens per window (window side w = sqrt(N))
    d: int          # per-head width d_h
    m: int          # landmarks
    dtypes: tuple   # storage types exercised ("f32", "bf16")
    recipe: str     # "iid" | "proj" | "smooth"
    seed: int
    description: str

    @property
    def window(self):
        w = int(round(self.N ** 0.5))
        assert w * w == self.N
        return w

    @property
    def units(self):
        return self.n_windows * self.heads

    def io_bytes(self, dtype):
        """Compulsory HBM traffic of one pass: read Q, K, V, write O."""
        e = 4 if dtype == "f32" else 2
        return 4 * self.units * self.N * self.d * e


CONFIGS = {
    "c1": Workload("c1", 64, 6, 64, 30, 16, ("f32",), "iid", 1001,
                   "64 windows x 6 heads, 8x8 windows (N=64), d_h=30, m=16; "
                   "Q,K,V i.i.d. N(0,1)"),
    "c2": Workload("c2", 1024, 6, 64, 30, 16, ("f32", "bf16"), "proj", 1002,
                   "SwinIR-like layer: 256x256 map, 8x8 windows -> 1024 windows x 6 heads, "
                   "N=64, d_h=30, m=16; Q,K,V = X W, X~N(0,1) width 180, W~N(0,1/180)"),
    "c3": Workload("c3", 4096, 1, 64, 32, 8, ("bf16",), "iid", 1003,
                   "Uformer-like shallow stage: 512x512 map, 8x8 windows -> 4096 windows x "
                   "1 head, N=64, d_h=32, m=8; Q,K,V i.i.d. N(0,1)"),
    "c4": Workload("c4", 1024, 6, 256, 30, 32, ("f32", "bf16"), "smooth", 1004,
                   "16x16 windows (N=256) on a 512x512x180 map, 1024 windows x 6 heads, "
                   "d_h=30, m=32; Q,K = shared Gaussian-filtered (sigma 2 px) N(0,1) field "
                   "+ N(0, 0.1^2) noise, V i.i.d. N(0,1)"),
    "c5": Workload("c5", 256, 8, 1024, 32, 64, ("bf16",), "iid", 1005,
                   "32x32 windows (N=1024) on a 512x512 map, 256 windows x 8 heads, d_h=32, "
                   "m=64; Q,K,V i.i.d. N(0,1)"),
}


def round_to(x, dtype):
    """Round float64 values to the storage type; return them as float64."""
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    if dtype == "f32":
        return x32.astype(np.float64)
    if dtype == "bf16":
        u = x32.view(np.uint32).astype(np.uint64)
        u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
        return u.astype(np.uint32).view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype}")


def partition(fmap, w, heads):
    """[H][W][C] feature map -> [windows][heads][w*w][C/heads]."""
    Hm, Wm, C = fmap.shape
    assert Hm % w == 0 and Wm % w == 0 and C % heads == 0
    x = fmap.reshape(Hm // w, w, Wm // w, w, heads, C // heads)
    x = x.transpose(0, 2, 4, 1, 3, 5)           # [wy][wx][h][ty][tx][c]
    return np.ascontiguousarray(x.reshape((Hm // w) * (Wm // w), heads, w * w, C // heads))


def _map_side(wl, n_windows):
    s = int(round(n_windows ** 0.5))
    if s * s != n_windows:
        raise ValueError("map recipes need a square number of windows")
    return s * wl.window


def generate(wl, dtype, n_windows=None, seed=None):
    """Q, K, V (float64 arrays holding dtype-rounded values) for a workload.

    ``n_windows`` shrinks the workload (the map recipes then use a smaller map
    of the same kind); ``seed`` overrides the workload's seed.
    """
    nw = wl.n_windows if n_windows is None else n_windows
    rng = np.random.default_rng(wl.seed if seed is None else seed)
    shape = (nw, wl.heads, wl.N, wl.d)
    if wl.recipe == "iid":
        q = rng.standard_normal(shape)
        k = rng.standard_normal(shape)
        v = rng.standard_normal(shape)
    elif wl.recipe == "proj":
        side = _map_side(wl, nw)
        C = wl.heads * wl.d
        x = rng.standard_normal((side, side, C))
        wq, wk, wv = (rng.standard_normal((C, C)) / np.sqrt(C) for _ in range(3))
        q = partition(x @ wq, wl.window, wl.heads)
        k = partition(x @ wk, wl.window, wl.heads)
        v = partition(x @ wv, wl.window, wl.heads)
    elif wl.recipe == "smooth":
        from scipy.ndimage import gaussian_filter
        side = _map_side(wl, nw)
        C = wl.heads * wl.d
        field = gaussian_filter(rng.standard_normal((side, side, C)), sigma=(2.0, 2.0, 0.0),
                                mode="reflect", truncate=4.0)
        q = partition(field + 0.1 * rng.standard_normal((side, side, C)), wl.window, wl.heads)
        k = partition(field + 0.1 * rng.standard_normal((side, side, C)), wl.window, wl.heads)
        v = partition(rng.standard_normal((side, side, C)), wl.window, wl.heads)
    else:
        raise ValueError(wl.recipe)
    return round_to(q, dtype), round_to(k, dtype), round_to(v, dtype)


def iid(shape, seed, dtype="f32", std=1.0):
    """Plain i.i.d. N(0, std^2) Q, K, V of an arbitrary [..., N, d] shape."""
    rng = np.random.default_rng(seed)
    return tuple(round_to(std * rng.standard_normal(shape), dtype) for _ in range(3))


def block_inputs(B, H, W, C, seed, dtype="f32", bias_std=0.02):
    """Feature map and synthetic weights of one window-attention block:
    x [B][H][W][C] ~ N(0, 1); W_qkv [C][3C] and W_proj [C][C] ~ N(0, 1/C)
    (the scale of a trained block's projections); biases ~ N(0, bias_std^2).
    Returns float64 arrays holding dtype-rounded values."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, H, W, C))
    w_qkv = rng.standard_normal((C, 3 * C)) / np.sqrt(C)
    b_qkv = bias_std * rng.standard_normal(3 * C)
    w_proj = rng.standard_normal((C, C)) / np.sqrt(C)
    b_proj = bias_std * rng.standard_normal(C)
    return tuple(round_to(a, dtype) for a in (x, w_qkv, b_qkv, w_proj, b_proj))
