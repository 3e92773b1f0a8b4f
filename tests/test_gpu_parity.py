"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Small cases are compared on every unit.  The full-size workloads run in the
launch configuration the benchmark times; the 64-token workloads are compared
on every unit, the larger ones on 256 strided units (first and last
included).  Bars (helpers.check): fp32 max-abs <= 1e-4; bf16 max-abs <= 2e-2
x RMS of the oracle output wherever the oracle's own bf16 rounding meets that
bar, and in every bf16 case the error beyond that rounding <= 2e-3 x RMS;
landmark maps bit-exact.
"""
import functools

import numpy as np
import pytest

import oracle
from paper_2506_08520_amd import binding as B
from paper_2506_08520_amd import workloads as W
from helpers import (torch_dtype, TOL, check, error, exact_bf16_allowance, sample_units, to_dev,
                     to_host)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

VARIANTS = [B.VARIANT_GENERIC, B.VARIANT_TILED]


def run(q, k, v, m, dtype, variant, iters=6, mode=0, scale=0.0):
    shape = q.shape
    tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
    opts = B.make_opts(pinv_iters=iters, landmark_mode=mode, scale=scale, variant=variant)
    o = B.nystra_attn_forward_ex(tq, tk, tv, m, opts=opts)
    torch.cuda.synchronize()
    out = to_host(o)
    assert out.shape == shape
    return out


def run_ws(q, k, v, m, dtype, variant, iters=6, mode=0, scale=0.0, workspace=None):
    """The workspace entry point (torch allocates the workspace it asks for)."""
    tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
    opts = B.make_opts(pinv_iters=iters, landmark_mode=mode, scale=scale, variant=variant)
    o = B.nystra_attn_forward_ws(tq, tk, tv, m, opts=opts, workspace=workspace)
    torch.cuda.synchronize()
    return to_host(o)


def check_config(got, ref, dtype, what):
    """The parity bar of helpers.check (kept under the name the tests use)."""
    return check(got, ref, dtype, what)


def need_variant(N, d, m, dtype, variant, mode=0):
    code = B.F32 if dtype == "f32" else B.BF16
    if variant == B.VARIANT_TILED:
        sel = B.nystra_select_variant(N, d, m, code, B.make_opts(landmark_mode=mode))
        if sel != B.VARIANT_TILED:
            pytest.skip("no MFMA-tiled kernel covers this shape; the generic kernel runs it")


SMALL = [("c1", "f32", 4), ("c2", "f32", 4), ("c2", "bf16", 4), ("c3", "bf16", 16),
         ("c4", "f32", 4), ("c4", "bf16", 4), ("c5", "bf16", 1)]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("cfg,dtype,nw", SMALL)
def test_config_shapes_all_units(cfg, dtype, nw, variant):
    wl = W.CONFIGS[cfg]
    need_variant(wl.N, wl.d, wl.m, dtype, variant)
    q, k, v = W.generate(wl, dtype, n_windows=nw)
    ref = oracle.forward(q, k, v, wl.m, iters=6, mode=0)
    got = run(q, k, v, wl.m, dtype, variant)
    check_config(got, ref, dtype, f"{cfg} {dtype} variant={variant}")


# (n_windows, heads, N, d, m, mode): ragged, degenerate and maximum shapes.
EDGE = [
    (3, 2, 36, 7, 6, 0),      # 6x6 window, 2x3 patches, odd width
    (2, 1, 9, 1, 9, 0),       # m = N, d = 1
    (2, 3, 64, 64, 64, 0),    # m = N = 64, widest head
    (1, 2, 4096, 64, 64, 0),  # largest window and head
    (5, 1, 64, 30, 1, 0),     # one landmark
    (2, 2, 100, 16, 25, 0),   # 10x10 window, 2x2 patches
    (2, 2, 48, 12, 12, 1),    # non-square N with 1-D segments
    (3, 1, 64, 32, 8, 1),     # 1-D segments at a config shape
    (1, 1, 1, 1, 1, 0),       # a single token: O = V
    (7, 3, 16, 5, 4, 0),      # tiny window, many units
    (2, 2, 256, 30, 16, 0),   # fewer landmarks at N = 256
    (1, 3, 1024, 30, 32, 0),  # m = 32 at N = 1024
    (2, 2, 64, 32, 32, 0),    # 1x2 patches, two landmark tiles at N = 64
    (2, 1, 144, 24, 36, 0),   # 12x12 window, 6x6 grid of 2x2 patches (three tiles)
    (1, 2, 4096, 32, 64, 0),  # largest window with four landmark tiles
    (1, 2, 1024, 16, 64, 1),  # 1-D segments at N = 1024
    (3, 2, 256, 8, 32, 1),    # 1-D segments, narrow head
    (2, 2, 240, 24, 48, 1),   # three landmark tiles, 1-D segments
    (2, 2, 384, 30, 24, 1),   # two landmark tiles, the second partly padding
    (2, 1, 49, 65, 7, 0),     # first width past 64 (odd)
    (2, 2, 64, 96, 16, 0),    # wide head at a config window
    (1, 2, 256, 128, 64, 0),  # widest head with the most landmarks (largest LDS)
    (1, 1, 1024, 128, 32, 1), # widest head, 1-D segments, long window
    (2, 1, 1024, 8, 64, 0),   # K pooled in the key pass (bf16): narrowest head
    (1, 2, 1024, 20, 64, 0),  # ... with overlapping feature chunks
    (1, 3, 1024, 24, 64, 0),  # ... and a spare column at d = 24
    (3, 2, 256, 8, 32, 0),    # ... 16 x 16 windows (one tile per image row)
    (2, 2, 256, 20, 32, 0),   # ... 16 x 16, overlapping chunks
]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", EDGE, ids=lambda s: "x".join(map(str, s)))
def test_edge_shapes(shape, dtype, variant):
    nw, h, N, d, m, mode = shape
    need_variant(N, d, m, dtype, variant, mode)
    q, k, v = W.iid((nw, h, N, d), seed=N * 131 + d * 7 + m + mode, dtype=dtype)
    ref = oracle.forward(q, k, v, m, iters=6, mode=mode)
    got = run(q, k, v, m, dtype, variant, mode=mode)
    check(got, ref, dtype, f"edge {shape} {dtype} variant={variant}")
    if N == 1:
        np.testing.assert_allclose(got, v, rtol=0, atol=1e-6 if dtype == "f32" else 1e-2)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("iters", [0, 1, 3, 5, 8])
def test_iteration_counts(iters, variant):
    """fp32 parity over the paper's iteration range and a little beyond (the
    float32 sensitivity at larger counts is documented by a CPU test)."""
    wl = W.CONFIGS["c1"]
    need_variant(wl.N, wl.d, wl.m, "f32", variant)
    q, k, v = W.generate(wl, "f32", n_windows=8)
    ref = oracle.forward(q, k, v, wl.m, iters=iters)
    got = run(q, k, v, wl.m, "f32", variant, iters=iters)
    check(got, ref, "f32", f"c1 K={iters} variant={variant}")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("iters", [0, 1, 5, 8])
def test_iteration_counts_large_window(iters, dtype, variant):
    wl = W.CONFIGS["c4"]
    need_variant(wl.N, wl.d, wl.m, dtype, variant)
    q, k, v = W.generate(wl, dtype, n_windows=4)
    ref = oracle.forward(q, k, v, wl.m, iters=iters)
    got = run(q, k, v, wl.m, dtype, variant, iters=iters)
    check(got, ref, dtype, f"c4 K={iters} {dtype} variant={variant}")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("iters", [0, 1, 5, 8])
def test_iteration_counts_pooled_keys(iters, variant):
    """32 x 32 windows with m = 64 in bf16: the kernel that pools K in its key
    pass, over the iteration range."""
    wl = W.CONFIGS["c5"]
    need_variant(wl.N, wl.d, wl.m, "bf16", variant)
    q, k, v = W.generate(wl, "bf16", n_windows=1)
    ref = oracle.forward(q, k, v, wl.m, iters=iters)
    got = run(q, k, v, wl.m, "bf16", variant, iters=iters)
    check(got, ref, "bf16", f"c5 K={iters} variant={variant}")


@pytest.mark.parametrize("variant", VARIANTS)
def test_custom_scale(variant):
    need_variant(64, 30, 16, "f32", variant)
    q, k, v = W.iid((4, 2, 64, 30), seed=77)
    ref = oracle.forward(q, k, v, 16, scale=0.05)
    got = run(q, k, v, 16, "f32", variant, scale=0.05)
    assert error(got, ref, "f32") <= TOL["f32"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,d,m,mode", [(64, 30, 16, 0), (64, 32, 8, 0), (256, 30, 32, 0),
                                        (1024, 32, 64, 0), (64, 30, 16, 1), (36, 7, 6, 0),
                                        (4096, 3, 64, 1)])
def test_landmark_pool(N, d, m, mode, dtype):
    q, k, _ = W.iid((3, 2, N, d), seed=N + m, dtype=dtype)
    qb, kb, mp = B.nystra_landmark_pool(to_dev(q, dtype), to_dev(k, dtype), m, mode=mode)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(mp.cpu().numpy(), oracle.landmark_map(N, m, mode))
    qb, kb = to_host(qb), to_host(kb)
    for u in range(6):
        w, h = divmod(u, 2)
        tr = oracle.unit_trace(q[w, h], k[w, h], q[w, h], m, iters=0, mode=mode)
        np.testing.assert_allclose(qb[w, h], tr["Qbar"], rtol=1e-6, atol=1e-6)
        np.testing.assert_allclose(kb[w, h], tr["Kbar"], rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(4, 6, 64, 30), (16, 1, 64, 32), (2, 3, 256, 30),
                                   (1, 4, 1024, 32), (3, 2, 36, 7), (2, 1, 1, 1),
                                   (1, 2, 4096, 8), (2, 2, 64, 64), (2, 1, 49, 65),
                                   (1, 2, 300, 128)])
def test_exact_kernel(shape, dtype):
    q, k, v = W.iid(shape, seed=sum(shape), dtype=dtype)
    ref = oracle.exact(q, k, v)
    o = B.nystra_exact_attn_forward(*(to_dev(x, dtype) for x in (q, k, v)))
    torch.cuda.synchronize()
    check(to_host(o), ref, dtype, f"exact {shape} {dtype}",
          allowance=exact_allowance(q, k, v, dtype))


def exact_allowance(q, k, v, dtype):
    """bf16 exact attention rounds its probabilities to bf16 (the bound of
    helpers.exact_bf16_allowance); fp32 has no allowance."""
    return exact_bf16_allowance(q, k, v, oracle.exact) if dtype == "bf16" else None


def test_exact_kernel_constant_values():
    q, k, _ = W.iid((2, 3, 256, 30), seed=5)
    v = np.ones_like(q)
    o = B.nystra_exact_attn_forward(*(to_dev(x, "f32") for x in (q, k, v)))
    torch.cuda.synchronize()
    np.testing.assert_allclose(to_host(o), 1.0, rtol=0, atol=1e-6)


# ------------------------------------------------- full-size workloads ----

@functools.lru_cache(maxsize=2)
def full_inputs(cfg, dtype):
    return W.generate(W.CONFIGS[cfg], dtype)


# (config, dtype, units compared): None = every unit.
FULL = [("c1", "f32", None), ("c2", "f32", None), ("c2", "bf16", None), ("c3", "bf16", None),
        ("c4", "f32", 256), ("c4", "bf16", 256), ("c5", "bf16", 256)]


@pytest.mark.parametrize("cfg,dtype,count,kernel",
                         [f + (kern,) for f in FULL for kern in ("nystrom", "exact")])
def test_full_size(cfg, dtype, count, kernel):
    """The full workload in the benchmark's launch configuration (AUTO
    variant, default options), PnP-Nystra and the exact-attention comparison
    kernel on the same inputs: every unit of the 64-token workloads, 256
    strided units (first and last included) of the larger ones."""
    wl = W.CONFIGS[cfg]
    q, k, v = full_inputs(cfg, dtype)
    tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
    if kernel == "nystrom":
        o = B.nystra_attn_forward(tq, tk, tv, wl.m)
    else:
        o = B.nystra_exact_attn_forward(tq, tk, tv)
    torch.cuda.synchronize()
    got = to_host(o).reshape(wl.units, wl.N, wl.d)
    del tq, tk, tv, o
    idx = sample_units(wl.units, count)
    assert idx[0] == 0 and idx[-1] == wl.units - 1
    sub = [x.reshape(-1, wl.N, wl.d)[idx] for x in (q, k, v)]
    if kernel == "nystrom":
        ref, allow = oracle.forward(*sub, wl.m), None
    else:
        ref, allow = oracle.exact(*sub), exact_allowance(*sub, dtype)
    check(got[idx], ref, dtype, f"full {cfg} {dtype} {kernel} on {len(idx)} of {wl.units} units",
          allowance=allow)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("order", ["rising", "falling"])
def test_running_max_order(order, dtype, variant):
    """Keys whose logits against every landmark rise (or fall) along the
    window: the row maximum m_U is reached in the last (or first) key tile, so
    a one-pass kernel rescales its partial sums at every tile (or never)."""
    nw, h, N, d, m = 2, 2, 256, 30, 32
    need_variant(N, d, m, dtype, variant)
    q, k, v = W.iid((nw, h, N, d), seed=7 + len(order), dtype=dtype)
    u = np.abs(q).mean(axis=2, keepdims=True)              # a direction Q-bar agrees with
    ramp = np.linspace(-1.0, 1.0, N)[None, None, :, None]
    if order == "falling":
        ramp = ramp[:, :, ::-1]
    k = W.round_to(k + 3.0 * ramp * np.sign(q.mean(axis=2, keepdims=True)) * (u > 0), dtype)
    ref = oracle.forward(q, k, v, m, iters=6, mode=0)
    got = run(q, k, v, m, dtype, variant)
    check(got, ref, dtype, f"running max {order} {dtype} variant={variant}")


# (m, K, N) grid of the sweep mode of bench.py, on small maps of its recipe
# (smooth field, d_h = 30): every (N, m) at K = 4 and the corners at other K.
SWEEP = ([(N, m, 4) for N in (64, 256, 1024, 4096) for m in (8, 16, 32, 64) if m <= N] +
         [(N, m, K) for N, m in ((64, 8), (4096, 64)) for K in (1, 3, 5, 6)])


@pytest.mark.parametrize("N,m,K", SWEEP)
def test_sweep_grid(N, m, K):
    w = int(round(N ** 0.5))
    wl = W.Workload("sweep", 4, 2, N, 30, m, ("f32",), "smooth", 2000 + N, f"{w}x{w} windows")
    q, k, v = W.generate(wl, "f32")
    ref = oracle.forward(q, k, v, m, iters=K, mode=0)
    got = run(q, k, v, m, "f32", B.VARIANT_AUTO, iters=K)
    err = error(got, ref, "f32")
    print(f"N={N} m={m} K={K}: max-abs {err:.3e}")
    assert err <= TOL["f32"]


# One window covering a whole map (global attention with pooled landmarks):
# (heads, N, d, m, mode, dtype).  d = 22 has no tiled kernel.
GLOBAL = [(2, 16384, 32, 64, 0, "f32"), (2, 16384, 32, 16, 1, "f32"), (1, 16384, 22, 64, 0, "f32"),
          (2, 65536, 32, 64, 0, "f32"), (2, 65536, 32, 64, 0, "bf16"), (2, 16384, 30, 32, 0, "bf16")]


@pytest.mark.parametrize("entry", ["ex", "ws"])
@pytest.mark.parametrize("shape", GLOBAL, ids=lambda s: "x".join(map(str, s)))
def test_global_window(shape, entry):
    """Both entry points with AUTO: the one-pass kernels through _ex, the
    token-split kernels (where they cover the shape) through _ws."""
    h, N, d, m, mode, dtype = shape
    q, k, v = W.iid((1, h, N, d), seed=N + d + m + mode, dtype=dtype)
    ref = oracle.forward(q, k, v, m, iters=6, mode=mode)
    if entry == "ex":
        got = run(q, k, v, m, dtype, B.VARIANT_AUTO, mode=mode)
    else:
        code = B.F32 if dtype == "f32" else B.BF16
        ws = B.nystra_attn_workspace_size(1, h, N, d, m, code, B.make_opts(landmark_mode=mode))
        assert (ws > 0) == (d % 4 == 0 or d == 30)
        got = run_ws(q, k, v, m, dtype, B.VARIANT_AUTO, mode=mode)
    check(got, ref, dtype, f"N={N} d={d} m={m} mode={mode} {dtype} {entry}")


# The token-split kernels forced through the workspace entry point:
# (n_windows, heads, N, d, m, mode, dtype).  N = 10000 has 25 x 25 patches
# (pieces and tiles straddle patch rows) and N % 32 == 16 (bf16 then takes the
# fp32 matrix-core path, and the last key chunk ends on an unpaired tile).
SPLIT = [(1, 2, 1024, 32, 16, 0, "f32"), (2, 3, 256, 30, 32, 0, "bf16"),
         (1, 1, 4096, 8, 64, 1, "f32"), (1, 2, 10000, 32, 16, 0, "f32"),
         (1, 2, 10000, 24, 16, 0, "bf16"), (1, 1, 2304, 16, 9, 0, "f32"),
         (1, 2, 16384, 32, 64, 0, "f32"), (1, 2, 20736, 30, 48, 0, "bf16"),
         (2, 1, 65536, 32, 64, 0, "bf16"), (1, 1, 65536, 16, 8, 1, "f32"),
         (16, 6, 64, 30, 16, 0, "f32"), (4, 8, 1024, 32, 64, 0, "bf16")]


@pytest.mark.parametrize("shape", SPLIT, ids=lambda s: "x".join(map(str, s)))
def test_split_kernels(shape):
    nw, h, N, d, m, mode, dtype = shape
    q, k, v = W.iid((nw, h, N, d), seed=3 * N + d + m, dtype=dtype)
    ref = oracle.forward(q, k, v, m, iters=6, mode=mode)
    got = run_ws(q, k, v, m, dtype, B.VARIANT_SPLIT, mode=mode)
    check(got, ref, dtype, f"split {shape}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("order", ["rising", "falling"])
def test_split_running_max_order(order, dtype):
    """The chunk maxima rise (or fall) from chunk to chunk, so the merge
    rescales every chunk record but the last (or first)."""
    nw, h, N, d, m = 1, 2, 4096, 32, 16
    q, k, v = W.iid((nw, h, N, d), seed=11 + len(order), dtype=dtype)
    u = np.abs(q).mean(axis=2, keepdims=True)
    ramp = np.linspace(-1.0, 1.0, N)[None, None, :, None]
    if order == "falling":
        ramp = ramp[:, :, ::-1]
    k = W.round_to(k + 3.0 * ramp * np.sign(q.mean(axis=2, keepdims=True)) * (u > 0), dtype)
    ref = oracle.forward(q, k, v, m, iters=6, mode=0)
    got = run_ws(q, k, v, m, dtype, B.VARIANT_SPLIT)
    check(got, ref, dtype, f"split running max {order} {dtype}")


def test_split_deterministic_and_workspace_reuse():
    """No atomics: repeated calls give identical bits, also when the workspace
    still holds the records of a different, larger problem."""
    q, k, v = W.iid((1, 2, 16384, 32), seed=5)
    tq, tk, tv = (to_dev(x, "f32") for x in (q, k, v))
    opts = B.make_opts(variant=B.VARIANT_SPLIT)
    big = B.nystra_attn_workspace_size(1, 4, 65536, 32, 64, B.F32, opts)
    ws = torch.full((big,), 0xFF, dtype=torch.uint8, device="cuda")   # NaN patterns
    a = B.nystra_attn_forward_ws(tq, tk, tv, 16, opts=opts, workspace=ws)
    qq, kk, vv = (to_dev(x, "f32") for x in W.iid((1, 4, 65536, 32), seed=6))
    B.nystra_attn_forward_ws(qq, kk, vv, 64, opts=opts, workspace=ws)
    b = B.nystra_attn_forward_ws(tq, tk, tv, 16, opts=opts, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    ref = oracle.forward(q, k, v, 16, iters=6, mode=0)
    assert error(to_host(a), ref, "f32") <= TOL["f32"]


# The head widths added for Dehazeformer-style models (d_h = 12, 16) and the
# other multiples of 4: every kernel family, both dtypes.
WIDTHS = [(64, 12, 16, "f32"), (64, 12, 16, "bf16"), (64, 20, 8, "bf16"), (64, 28, 16, "f32"),
          (256, 12, 32, "bf16"), (256, 20, 32, "f32"), (1024, 28, 64, "bf16"),
          (1024, 12, 16, "f32")]


@pytest.mark.parametrize("N,d,m,dtype", WIDTHS)
def test_new_head_widths(N, d, m, dtype):
    code = B.F32 if dtype == "f32" else B.BF16
    assert B.nystra_select_variant(N, d, m, code) == B.VARIANT_TILED
    q, k, v = W.iid((2, 3, N, d), seed=N + d + m, dtype=dtype)
    ref = oracle.forward(q, k, v, m, iters=6, mode=0)
    for name, got in (("tiled", run(q, k, v, m, dtype, B.VARIANT_TILED)),
                      ("split", run_ws(q, k, v, m, dtype, B.VARIANT_SPLIT))):
        check(got, ref, dtype, f"width {d} N={N} m={m} {dtype} {name}")
    ex = to_host(B.nystra_exact_attn_forward(*(to_dev(x, dtype) for x in (q, k, v))))
    check(ex, oracle.exact(q, k, v), dtype, f"width {d} N={N} {dtype} exact",
          allowance=exact_allowance(q, k, v, dtype))


def test_exact_kernel_long_window():
    """Exact attention at N = 8192 (V^T no longer fits the LDS stage)."""
    q, k, v = W.iid((1, 1, 8192, 32), seed=8192, dtype="f32")
    ref = oracle.exact(q, k, v)
    got = to_host(B.nystra_exact_attn_forward(*(to_dev(x, "f32") for x in (q, k, v))))
    assert error(got, ref, "f32") <= TOL["f32"]


# --------------------------------------------------------- behaviour ----

def test_deterministic_and_stream_independent():
    q, k, v = W.generate(W.CONFIGS["c2"], "f32", n_windows=16)
    tq, tk, tv = (to_dev(x, "f32") for x in (q, k, v))
    a = B.nystra_attn_forward(tq, tk, tv, 16)
    b = B.nystra_attn_forward(tq, tk, tv, 16)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        c = B.nystra_attn_forward(tq, tk, tv, 16, stream=s)
    s.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(a, c)


def test_output_untouched_on_validation_error():
    q, k, v = (to_dev(x, "f32") for x in W.iid((2, 2, 64, 30), seed=3))
    o = torch.full_like(q, 7.0)
    with pytest.raises(B.NystraError) as e:
        B.nystra_attn_forward(q, k, v, 3, out=o)   # no pooling grid for m = 3
    assert e.value.status == 2
    with pytest.raises(B.NystraError):
        B.nystra_attn_forward_ex(q, k, v, 16, opts=B.make_opts(pinv_iters=99), out=o)
    torch.cuda.synchronize()
    assert bool((o == 7.0).all())


# (dtype, element offset, does a tiled kernel take it): fp32 tiled kernels take
# any element alignment; bf16 needs 4-byte aligned tensors (2 bytes: the generic
# kernel runs).
ALIGN = [("f32", 1, True), ("bf16", 1, False), ("f32", 4, True), ("bf16", 8, True)]


@pytest.mark.parametrize("dtype,offset,tiled", ALIGN)
def test_element_aligned_tensors(dtype, offset, tiled):
    """Tensors offset from their allocation: a forced tiled launch runs when a
    tiled kernel can take the alignment and is refused before touching O
    otherwise; AUTO always runs, and results match the oracle."""
    wl = W.CONFIGS["c2"]
    q, k, v = W.generate(wl, dtype, n_windows=4)
    ref = oracle.forward(q, k, v, wl.m, iters=6, mode=0)
    n = q.size
    flat = [torch.zeros(n + offset, dtype=torch_dtype(dtype), device="cuda") for _ in range(4)]
    views = [f[offset:].view(q.shape) for f in flat]
    for view, x in zip(views[:3], (q, k, v)):
        view.copy_(to_dev(x, dtype))
    o = views[3]
    o.fill_(7.0)
    forced = B.make_opts(variant=B.VARIANT_TILED)
    if tiled:
        B.nystra_attn_forward_ex(*views[:3], wl.m, opts=forced, out=o)
        torch.cuda.synchronize()
        check_config(to_host(o), ref, dtype, f"c2 {dtype} offset {offset} tiled")
        o.fill_(7.0)
    else:
        with pytest.raises(B.NystraError) as e:
            B.nystra_attn_forward_ex(*views[:3], wl.m, opts=forced, out=o)
        assert e.value.status == 6
        torch.cuda.synchronize()
        assert bool((o == 7.0).all())
    B.nystra_attn_forward_ex(*views[:3], wl.m, opts=B.make_opts(), out=o)
    torch.cuda.synchronize()
    check_config(to_host(o), ref, dtype, f"c2 {dtype} offset {offset} auto")


def test_empty_batch_is_noop():
    q = torch.empty((0, 6, 64, 30), device="cuda")
    o = B.nystra_attn_forward(q, q, q, 16)
    assert o.numel() == 0


# The small-window kernel launches one-wave workgroups below 1024 units and
# four-wave workgroups from 1024 on (LDS sized by the workgroup); both sides of
# that switch, every unit compared, for both fixed pooling grids.
@pytest.mark.parametrize("units,heads,d,m,dtype",
                         [(1020, 6, 30, 16, "f32"), (1026, 6, 30, 16, "f32"),
                          (1023, 1, 32, 8, "bf16"), (1025, 1, 32, 8, "bf16")])
def test_small_kernel_launch_geometry(units, heads, d, m, dtype):
    assert units % heads == 0
    shape = (units // heads, heads, 64, d)
    assert B.nystra_select_variant(64, d, m, B.F32 if dtype == "f32" else B.BF16) == B.VARIANT_TILED
    q, k, v = W.iid(shape, seed=units + d, dtype=dtype)
    ref = oracle.forward(q, k, v, m, iters=6, mode=0)
    got = run(q, k, v, m, dtype, B.VARIANT_TILED)
    check_config(got, ref, dtype, f"{units} units {dtype}")
