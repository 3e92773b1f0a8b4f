"""Host-side checks of the C ABI: exports, the host landmark map, and every
argument-validation path.  No call here reaches a kernel launch, so these run
without a GPU."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from paper_2506_08520_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nystra.h")

OK, ENULL, ESHAPE, EDTYPE, EALIGN, EOVERLAP, EUNSUP, EHIP, EARG, EWS = range(10)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nystra_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return B.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 9
    assert sorted(B.EXPORTS) == names
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (nystra_\w+)", out))
    for n in names:
        assert n in exported, n
        assert hasattr(L, n)


def test_library_links_no_torch():
    out = subprocess.run(["ldd", B.LIB_PATH], capture_output=True, text=True).stdout
    # library names only: the load addresses ldd prints are random hex
    names = [line.split("(")[0].split("=>")[-1].strip() for line in out.splitlines()]
    assert names and "libamdhip64" in " ".join(names)
    assert not any("torch" in n or "c10" in n for n in names), names


@pytest.mark.parametrize("N,m,mode", [(64, 16, 0), (64, 8, 0), (256, 32, 0), (1024, 64, 0),
                                      (64, 16, 1), (64, 8, 1), (256, 32, 1), (1024, 64, 1),
                                      (36, 6, 0), (4096, 64, 0), (9, 9, 0), (16, 1, 0),
                                      (4096, 64, 1), (100, 25, 0), (24, 6, 1)])
def test_host_map_bit_exact_vs_oracle(N, m, mode):
    np.testing.assert_array_equal(B.nystra_landmark_map(N, m, mode),
                                  oracle.landmark_map(N, m, mode))


def test_host_map_matches_hand_written(golden_maps):
    for (N, m, mode), grid in golden_maps.items():
        np.testing.assert_array_equal(B.nystra_landmark_map(N, m, mode), grid)


def test_host_map_rejects_what_the_oracle_rejects():
    for N, m, mode in [(63, 7, 0), (64, 3, 0), (64, 5, 1), (50, 5, 0), (64, 65, 0)]:
        with pytest.raises(B.NystraError) as e:
            B.nystra_landmark_map(N, m, mode)
        assert e.value.status == ESHAPE
    with pytest.raises(B.NystraError):
        B.nystra_landmark_map(64, 16, 9)


# A fake, well-aligned device address: validation rejects every call below
# before anything would touch it.
P = 1 << 20


def fwd(L, q=P, k=P + (1 << 24), v=P + (2 << 24), o=P + (3 << 24), W=2, H=3, N=64, d=30, m=16,
        dtype=0, opts=None):
    po = ctypes.byref(opts) if opts is not None else None
    return L.nystra_attn_forward_ex(q, k, v, o, W, H, N, d, m, dtype, po, None)


def test_forward_validation(L):
    assert fwd(L, dtype=2) == EDTYPE
    assert fwd(L, dtype=-1) == EDTYPE
    for kw in [dict(N=0), dict(N=(1 << 20) + 1), dict(d=0), dict(d=129), dict(m=0), dict(m=65, N=4096),
               dict(m=65), dict(W=-1), dict(H=-2), dict(N=63, m=7), dict(N=64, m=3),
               dict(W=1 << 16, H=1 << 16), dict(W=1 << 24, H=1), dict(W=1 << 23, H=2),
               dict(W=(1 << 23) + 1, H=2)]:
        assert fwd(L, **kw) == ESHAPE, kw
    seg = B.make_opts(landmark_mode=1)
    assert fwd(L, N=64, m=5, opts=seg) == ESHAPE
    for o in [B.make_opts(pinv_iters=-1), B.make_opts(pinv_iters=65), B.make_opts(landmark_mode=2),
              B.make_opts(variant=4), B.make_opts(variant=-1), B.make_opts(scale=float("nan")),
              B.make_opts(scale=float("inf"))]:
        assert fwd(L, opts=o) == EARG
    # the token-split kernels need a workspace, which this entry point lacks
    assert fwd(L, opts=B.make_opts(variant=B.VARIANT_SPLIT)) == EUNSUP
    assert fwd(L, q=None) == ENULL
    assert fwd(L, o=None) == ENULL
    assert fwd(L, q=P + 2) == EALIGN
    assert fwd(L, o=P + (3 << 24) + 2) == EALIGN
    assert fwd(L, dtype=1, v=P + (2 << 24) + 1) == EALIGN
    # bf16 needs only 2-byte alignment: an odd-halfword O is fine for alignment,
    # so the overlap check is what fails here
    assert fwd(L, dtype=1, o=P + 2) == EOVERLAP
    assert fwd(L, o=P + 100) == EOVERLAP
    assert fwd(L, o=P + (1 << 24) - 4) == EOVERLAP   # tail of Q meets head of O
    # empty batches are a no-op whatever the pointers
    assert fwd(L, W=0, q=None, k=None, v=None, o=None) == OK
    assert fwd(L, H=0, q=None, k=None, v=None, o=None) == OK


def test_default_forward_validation(L):
    r = L.nystra_attn_forward(P, P + (1 << 24), P + (2 << 24), None, 2, 3, 64, 30, 16, 0, None)
    assert r == ENULL
    r = L.nystra_attn_forward(P, P, P, P, 0, 3, 64, 30, 16, 0, None)
    assert r == OK


def test_exact_validation(L):
    f = L.nystra_exact_attn_forward
    q, k, v, o = P, P + (1 << 24), P + (2 << 24), P + (3 << 24)
    assert f(q, k, v, o, 2, 3, 64, 30, 7, 0.0, None) == EDTYPE
    assert f(q, k, v, o, 2, 3, 0, 30, 0, 0.0, None) == ESHAPE
    assert f(q, k, v, o, 2, 3, 64, 129, 0, 0.0, None) == ESHAPE
    assert f(q, k, v, o, 2, 3, 64, 30, 0, float("nan"), None) == EARG
    assert f(None, k, v, o, 2, 3, 64, 30, 0, 0.0, None) == ENULL
    assert f(q, k, v, q + 8, 2, 3, 64, 30, 0, 0.0, None) == EOVERLAP
    assert f(q, k, v, o + 1, 2, 3, 64, 30, 1, 0.0, None) == EALIGN
    assert f(None, None, None, None, 0, 3, 64, 30, 0, 0.0, None) == OK


def test_landmark_pool_validation(L):
    f = L.nystra_landmark_pool
    q, k, qb, kb = P, P + (1 << 24), P + (2 << 24), P + (3 << 24)
    assert f(q, k, qb, kb, None, 2, 3, 64, 30, 16, 4, 0, None) == EDTYPE
    assert f(q, k, qb, kb, None, 2, 3, 64, 30, 3, 0, 0, None) == ESHAPE
    assert f(q, k, qb, kb, None, 2, 3, 64, 30, 16, 0, 5, None) == EARG
    assert f(q, k, None, kb, None, 2, 3, 64, 30, 16, 0, 0, None) == ENULL
    assert f(q, k, qb + 2, kb, None, 2, 3, 64, 30, 16, 1, 0, None) == EALIGN
    assert f(q, k, qb, kb, P + (4 << 24) + 2, 2, 3, 64, 30, 16, 0, 0, None) == EALIGN
    assert f(q, k, q + 16, kb, None, 2, 3, 64, 30, 16, 0, 0, None) == EOVERLAP
    assert f(q, k, qb, qb + 64, None, 2, 3, 64, 30, 16, 0, 0, None) == EOVERLAP
    assert f(None, None, None, None, None, 0, 3, 64, 30, 16, 0, 0, None) == OK


def test_status_strings_and_opts(L):
    for s in range(10):
        assert B.nystra_status_str(s) and B.nystra_status_str(s) != "unknown status"
    assert B.nystra_status_str(99) == "unknown status"
    o = B.nystra_default_opts()
    assert (o.pinv_iters, o.landmark_mode, o.scale, o.variant) == (6, 0, 0.0, 0)
    assert L.nystra_default_opts(None) == ENULL
    assert L.nystra_last_error() == b""


def test_variant_selection():
    # tiled head widths: multiples of 4 from 8 to 32, and 30
    for d in range(1, 129):
        tiled = 8 <= d <= 32 and (d % 4 == 0 or d == 30)
        sel = B.nystra_select_variant(256, d, 16)
        assert sel == (B.VARIANT_TILED if tiled else B.VARIANT_GENERIC), d
    g = B.VARIANT_GENERIC
    assert B.nystra_select_variant(64, 30, 16, opts=B.make_opts(variant=g)) == g
    assert B.nystra_select_variant(49, 64, 7) in (B.VARIANT_GENERIC, B.VARIANT_TILED)
    with pytest.raises(B.NystraError):
        B.nystra_select_variant(63, 30, 7)
    with pytest.raises(B.NystraError):
        B.nystra_select_variant(64, 30, 16, opts=B.make_opts(pinv_iters=-3))



def ws_size(W, H, N, d, m, dtype=0, **opts):
    return B.nystra_attn_workspace_size(W, H, N, d, m, dtype, B.make_opts(**opts))


def test_workspace_size():
    split = B.VARIANT_SPLIT
    # global window, few units: AUTO takes the token-split kernels
    big = ws_size(1, 6, 1 << 18, 32, 64)
    assert 0 < big < 64 << 20
    assert ws_size(1, 6, 1 << 18, 32, 64, 1) == big   # fp32 records for either dtype
    # one workgroup per unit fills the GPU: no workspace
    assert ws_size(1024, 6, 64, 30, 16) == 0
    assert ws_size(256, 8, 1024, 32, 64) == 0
    # forced: any supported shape, sized from the same plan
    assert ws_size(1024, 6, 64, 30, 16, variant=split) > 0
    assert ws_size(1, 6, 1 << 18, 32, 64, variant=split) == big
    assert ws_size(1, 6, 1 << 18, 32, 64, variant=B.VARIANT_TILED) == 0
    assert ws_size(1, 6, 1 << 18, 32, 64, variant=B.VARIANT_GENERIC) == 0
    # more tokens, more chunk records
    assert ws_size(1, 2, 1 << 16, 32, 64) < ws_size(1, 2, 1 << 18, 32, 64)
    assert ws_size(0, 6, 1 << 18, 32, 64) == 0
    # shapes the token-split kernels do not cover
    for args in [(1, 1, 16384, 22, 64), (1, 1, 100, 32, 4), (1, 1, 16384, 48, 64)]:
        with pytest.raises(B.NystraError) as e:
            ws_size(*args, variant=split)
        assert e.value.status == EUNSUP
        assert ws_size(*args) == 0   # AUTO falls back to the other kernels
    with pytest.raises(B.NystraError) as e:
        ws_size(1, 1, 63, 32, 7)
    assert e.value.status == ESHAPE
    assert B.lib().nystra_attn_workspace_size(1, 1, 4096, 32, 16, 0, None, None) == ENULL


def test_forward_ws_validation(L):
    q, k, v, o = P, P + (1 << 24), P + (2 << 24), P + (3 << 24)
    ws = P + (4 << 24)
    N, d, m = 4096, 32, 16
    need = ws_size(1, 2, N, d, m)
    assert need > 0
    opts = B.make_opts()

    def f(ws=ws, nbytes=need, q=q, o=o, N=N, opts=opts):
        return L.nystra_attn_forward_ws(q, k, v, o, 1, 2, N, d, m, 0, ctypes.byref(opts), ws,
                                        nbytes, None)

    # every failure below is detected before anything is enqueued
    assert f(ws=None) == EWS
    assert f(nbytes=need - 1) == EWS
    assert f(ws=ws + 128) == EWS          # not 256-byte aligned
    assert f(ws=q + 256) == EWS           # overlaps Q
    assert f(ws=o - 1024) == EWS          # runs into O
    assert f(q=None) == ENULL
    assert f(o=q + 64) == EOVERLAP
    assert f(N=4095) == ESHAPE
    assert f(opts=B.make_opts(variant=5)) == EARG
    # the token-split kernels store O in 16-byte pieces
    assert f(opts=B.make_opts(variant=B.VARIANT_SPLIT), o=o + 4) == EUNSUP
    assert f(opts=B.make_opts(variant=B.VARIANT_SPLIT), N=4096 + 16) == ESHAPE  # no 2-D grid
    assert L.nystra_attn_forward_ws(None, None, None, None, 0, 2, N, d, m, 0, None, None, 0,
                                    None) == OK


def bshape(**kw):
    d = dict(batch=1, height=16, width=16, channels=96, heads=3, window=8, shift=0)
    d.update(kw)
    return B.BlockShape(*(d[k] for k in ("batch", "height", "width", "channels", "heads",
                                         "window", "shift")))


def test_noalloc_rejects_more_than_its_scratch(L):
    """The allocation-free entry point refuses, before any launch, a call
    whose token-split workspace exceeds its static array."""
    opts = B.make_opts(variant=B.VARIANT_SPLIT)
    W_, H_, N_, d_, m_ = 16, 6, 262144, 30, 64
    assert B.nystra_attn_workspace_size(W_, H_, N_, d_, m_, 0, opts) > B.STATIC_SCRATCH_BYTES
    assert B.nystra_attn_workspace_size(1, 6, N_, d_, m_, 0, opts) <= B.STATIC_SCRATCH_BYTES
    step = 1 << 33   # fake, disjoint, aligned device addresses
    q, k, v, o = (ctypes.c_void_p(step * (i + 1)) for i in range(4))
    f = L.nystra_attn_forward_noalloc
    assert f(q, k, v, o, W_, H_, N_, d_, m_, 0, ctypes.byref(opts), None) == EWS
    assert b"NYSTRA_STATIC_SCRATCH_BYTES" in L.nystra_last_error()
    # the other validation paths are those of nystra_attn_forward_ws
    assert f(None, k, v, o, 1, 6, N_, d_, m_, 0, ctypes.byref(opts), None) == ENULL
    assert f(q, k, v, o, 1, 6, N_, 129, m_, 0, ctypes.byref(opts), None) == ESHAPE
    assert f(q, k, v, o, 0, 6, N_, d_, m_, 0, None, None) == OK


def packed_weight_bytes(C, ncols, bf16):
    """The GEMM's packed image of a [C][ncols] weight: one LDS tile image per
    64 columns (fp32 [KP][68] words, bf16 [64][KP + 8] halves), KP the
    contraction padded to 32, 64, 128, 192 or 256; none past C = 256."""
    kp = next((x for x in (32, 64, 128, 192, 256) if C <= x), None)
    if kp is None:
        return 0
    words = 32 * (kp + 8) if bf16 else kp * 68
    return -(-ncols // 64) * words * 4


def test_block_workspace_size():
    one = 16 * 16 * 96 * 4                      # one of Q, K, V, O in fp32 (256-byte multiple)
    pk32 = packed_weight_bytes(96, 288, False) + packed_weight_bytes(96, 96, False)
    pk16 = packed_weight_bytes(96, 288, True) + packed_weight_bytes(96, 96, True)
    assert pk32 % 256 == 0 and pk16 % 256 == 0
    assert B.nystra_block_workspace_size(bshape(), 16) == 4 * one + pk32
    assert B.nystra_block_workspace_size(bshape(), 16, B.BF16) == 2 * one + pk16
    assert B.nystra_block_workspace_size(bshape(shift=4), 16, attention=B.BLOCK_EXACT) == 4 * one + pk32
    assert B.nystra_block_workspace_size(bshape(batch=0), 16) == 0
    # a whole-map window takes the token-split attention, whose workspace comes on top
    glob = bshape(height=128, width=128, channels=64, heads=2, window=128)
    assert B.nystra_block_workspace_size(glob, 64) > 4 * 128 * 128 * 64 * 4
    for kw, status in [(dict(window=6), ESHAPE), (dict(shift=8), ESHAPE), (dict(shift=-1), ESHAPE),
                       (dict(channels=100), ESHAPE), (dict(heads=0), ESHAPE),
                       (dict(channels=4104, heads=3), ESHAPE), (dict(height=0), ESHAPE)]:
        with pytest.raises(B.NystraError) as e:
            B.nystra_block_workspace_size(bshape(**kw), 16)
        assert e.value.status == status, kw
    for args, status in [((16, 5), EDTYPE), ((3, 0), ESHAPE)]:
        with pytest.raises(B.NystraError) as e:
            B.nystra_block_workspace_size(bshape(), *args)
        assert e.value.status == status
    with pytest.raises(B.NystraError) as e:
        B.nystra_block_workspace_size(bshape(), 16, attention=2)
    assert e.value.status == EARG
    n = ctypes.c_size_t(0)
    assert B.lib().nystra_block_workspace_size(None, 16, 0, None, 0, ctypes.byref(n)) == ENULL
    assert B.lib().nystra_block_workspace_size(ctypes.byref(bshape()), 16, 0, None, 0,
                                               None) == ENULL


def test_block_forward_validation(L):
    s = bshape()
    need = B.nystra_block_workspace_size(s, 16)
    x, wq, wp, y, ws = P, P + (1 << 24), P + (2 << 24), P + (3 << 24), P + (4 << 24)

    def f(x=x, wq=wq, bq=None, wp=wp, bp=None, y=y, ws=ws, nb=need, s=s, dtype=0):
        return L.nystra_block_forward(x, wq, bq, wp, bp, y, ctypes.byref(s), 16, dtype, None, 0,
                                      ws, nb, None)

    assert f(x=None) == ENULL
    assert f(wp=None) == ENULL
    assert f(x=x + 2) == EALIGN
    assert f(bq=wq + (1 << 20) + 2) == EALIGN
    assert f(y=x + 64) == EOVERLAP
    assert f(y=wq - 256) == EOVERLAP          # Y's tail meets W_qkv
    assert f(ws=None) == EWS
    assert f(nb=need - 1) == EWS
    assert f(ws=ws + 64) == EWS
    assert f(ws=y) == EWS
    assert f(s=bshape(batch=0), x=None, y=None, ws=None) == OK


def test_block_packed_size():
    for C in (32, 96, 180, 256):
        for bf16 in (False, True):
            want = packed_weight_bytes(C, 3 * C, bf16) + packed_weight_bytes(C, C, bf16)
            got = B.nystra_block_packed_size(C, B.BF16 if bf16 else B.F32)
            assert got == want, (C, bf16)
            # the block workspace reserves the same bytes for the per-call packing
            heads = C // 16 if C % 16 == 0 else 6
            plain = B.nystra_block_workspace_size(bshape(channels=C, heads=heads), 16,
                                                  B.BF16 if bf16 else B.F32)
            assert plain >= got
    assert B.nystra_block_packed_size(288) == 0       # the block reads wider weights as given
    n = ctypes.c_size_t(0)
    assert B.lib().nystra_block_packed_size(96, 0, None) == ENULL
    assert B.lib().nystra_block_packed_size(96, 7, ctypes.byref(n)) == EDTYPE
    assert B.lib().nystra_block_packed_size(0, 0, ctypes.byref(n)) == ESHAPE
    assert B.lib().nystra_block_packed_size(4097, 0, ctypes.byref(n)) == ESHAPE


def test_block_pack_and_packed_forward_validation(L):
    need = B.nystra_block_packed_size(96)
    wq, wp, pk = P, P + (1 << 24), P + (2 << 24)
    pack = L.nystra_block_pack_weights
    assert pack(None, wp, 96, 0, pk, need, None) == ENULL
    assert pack(wq, wp, 96, 0, None, need, None) == ENULL
    assert pack(wq + 2, wp, 96, 0, pk, need, None) == EALIGN
    assert pack(wq, wp, 96, 0, pk + 64, need, None) == EALIGN
    assert pack(wq, wp, 96, 0, pk, need - 1, None) == EWS
    assert pack(wq, wp, 96, 0, wp - 256, need, None) == EOVERLAP   # the image meets W_proj
    assert pack(wq, wp, 96, 5, pk, need, None) == EDTYPE
    assert pack(None, None, 288, 0, None, 0, None) == OK            # nothing to pack past 256

    s = bshape()
    nb = B.nystra_block_workspace_size(s, 16)
    x, y, ws = P + (3 << 24), P + (4 << 24), P + (5 << 24)

    def f(packed=pk, pb=need, y=y, ws=ws, s=s):
        return L.nystra_block_forward_packed(x, wq, None, wp, None, packed, pb, y,
                                             ctypes.byref(s), 16, 0, None, 0, ws, nb, None)

    assert f(packed=None) == ENULL
    assert f(pb=need - 1) == EWS
    assert f(packed=pk + 64) == EALIGN
    assert f(packed=y) == EOVERLAP
    assert f(packed=ws) == EOVERLAP
    assert f(ws=ws + 64) == EWS                  # the other checks are nystra_block_forward's
    assert f(s=bshape(batch=0), packed=None) == OK
