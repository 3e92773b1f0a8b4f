"""GPU parity of the window-attention block (nystra_block_forward) against
the float64 block oracle: projections, window partition with cyclic shift,
head split and merge, window reverse, around PnP-Nystra or exact attention.
Bars (helpers.check): fp32 max-abs <= 1e-4.  bf16: max-abs <= 2e-2 x RMS
wherever the oracle's own bf16 rounding of Y meets that bar, and the error
beyond the rounding of Y <= BLOCK_BEYOND_BF16 = 2e-2 x RMS.  The oracle's Y is
taken before its own final rounding, so that the bars see the GPU's rounding
of Y as a rounding.  A bf16 block stores three times (Q/K/V, the attention
output, Y) as a bf16 model does, and the block oracle rounds Q/K/V and the
attention output at the same places -- but from float64 values, where the GPU
rounds fp32 GEMM and attention results.  An element whose value
lies within that fp32 error of a bf16 rounding midpoint is stored one bf16
ulp apart on the two sides, and such flips of intermediate tensors carry into
Y (measured: 0.66-1.4e-2 of RMS beyond the rounding of Y).  The kernels' own
precision is held to the 2e-3 bar by the operator tests, where the inputs are
stored exactly."""
import numpy as np
import pytest

from oracle import block as OB
from paper_2506_08520_amd import binding as B
from paper_2506_08520_amd import workloads as W
from helpers import TOL, check, error, to_dev, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


BLOCK_BEYOND_BF16 = 2e-2


def run_block(inputs, heads, window, shift, m, dtype, attention, mode=0, iters=6, nobias=False):
    x, wq, bq, wp, bp = (to_dev(a, dtype) for a in inputs)
    if nobias:
        bq = bp = None
    opts = B.make_opts(pinv_iters=iters, landmark_mode=mode)
    att = B.BLOCK_NYSTROM if attention == "nystrom" else B.BLOCK_EXACT
    y = B.nystra_block_forward(x, wq, bq, wp, bp, heads, window, shift=shift, m=m, opts=opts,
                               attention=att)
    torch.cuda.synchronize()
    return to_host(y)


# (B, H, W, C, heads, window, shift, m, dtype, attention)
CASES = [
    (1, 32, 32, 180, 6, 8, 0, 16, "f32", "nystrom"),    # SwinIR-shaped (c2 layer, smaller map)
    (1, 32, 32, 180, 6, 8, 4, 16, "f32", "nystrom"),    # shifted windows
    (2, 24, 16, 180, 6, 8, 4, 16, "bf16", "nystrom"),
    (1, 32, 32, 32, 1, 8, 4, 8, "bf16", "nystrom"),     # Uformer-shaped (c3)
    (1, 32, 48, 180, 6, 16, 8, 32, "f32", "nystrom"),   # 16 x 16 windows (c4)
    (1, 64, 64, 256, 8, 32, 16, 64, "bf16", "nystrom"), # 32 x 32 windows (c5)
    # 240 tokens: ragged row tile, d_h = 8.  (m = 4 here is so ill-conditioned
    # that fp32-sized input noise moves the float64 oracle by 4e-5 at outputs
    # of 19; m = 8 is not.)
    (1, 12, 20, 24, 3, 4, 2, 8, "f32", "nystrom"),
    (1, 16, 16, 66, 3, 8, 3, 16, "f32", "nystrom"),     # d_h = 22: generic attention kernel
    (1, 32, 32, 24, 2, 8, 4, 16, "bf16", "nystrom"),    # Dehazeformer-shaped: d_h = 12
    (2, 16, 16, 96, 3, 8, 4, 0, "f32", "exact"),
    (1, 16, 16, 180, 6, 16, 8, 0, "bf16", "exact"),
    (1, 64, 64, 64, 2, 64, 0, 64, "f32", "nystrom"),    # one window per map: token-split path
    (1, 64, 64, 64, 2, 64, 32, 16, "bf16", "nystrom"),
    (1, 16, 16, 256, 2, 8, 4, 16, "f32", "nystrom"),    # d_h = 128 (widest head)
    (1, 16, 24, 192, 2, 8, 0, 8, "bf16", "nystrom"),    # d_h = 96
    # odd d_h (15) and 135 QKV columns: the GEMM epilogue stores single columns
    (1, 16, 16, 45, 3, 8, 4, 16, "f32", "nystrom"),
    (1, 16, 16, 45, 3, 8, 4, 16, "bf16", "nystrom"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_block_parity(case):
    Bn, H, Wd, C, heads, w, s, m, dtype, att = case
    inputs = W.block_inputs(Bn, H, Wd, C, seed=H * Wd + C + s, dtype=dtype)
    ref = OB.block_forward(*inputs, heads=heads, window=w, shift=s, m=max(m, 1), attention=att,
                           dtype=dtype, round_output=False)
    got = run_block(inputs, heads, w, s, m, dtype, att)
    check(got, ref, dtype, f"block {case}", beyond_bar=BLOCK_BEYOND_BF16)


def test_block_without_biases_and_segment_pooling():
    inputs = W.block_inputs(1, 16, 16, 96, seed=77, dtype="f32")
    x, wq, _, wp, _ = inputs
    zq, zp = np.zeros(3 * 96), np.zeros(96)
    ref = OB.block_forward(x, wq, zq, wp, zp, heads=3, window=8, shift=2, m=8, mode=1)
    got = run_block(inputs, 3, 8, 2, 8, "f32", "nystrom", mode=1, nobias=True)
    assert error(got, ref, "f32") <= TOL["f32"]


def test_block_deterministic():
    inputs = W.block_inputs(1, 32, 32, 180, seed=5, dtype="f32")
    a = run_block(inputs, 6, 8, 4, 16, "f32", "nystrom")
    b = run_block(inputs, 6, 8, 4, 16, "f32", "nystrom")
    assert np.array_equal(a, b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_block_weights_repacked_every_call(dtype):
    """The GEMMs read the weights from a packed copy in the workspace, written
    by each call: a second call with other weights on the same workspace must
    give the second weights' block, not the first's."""
    C, heads, w, s, m = 96, 3, 8, 4, 16
    first = W.block_inputs(1, 16, 16, C, seed=11, dtype=dtype)
    second = W.block_inputs(1, 16, 16, C, seed=12, dtype=dtype)
    x = to_dev(first[0], dtype)
    shape = B.BlockShape(1, 16, 16, C, heads, w, s)
    code = B.F32 if dtype == "f32" else B.BF16
    ws = torch.empty(B.nystra_block_workspace_size(shape, m, code), dtype=torch.uint8,
                     device="cuda")
    ys = []
    for inp in (first, second):
        wq, bq, wp, bp = (to_dev(a, dtype) for a in inp[1:])
        ys.append(to_host(B.nystra_block_forward(x, wq, bq, wp, bp, heads, w, shift=s, m=m,
                                                 workspace=ws)))
    torch.cuda.synchronize()
    for seed, inp, y in zip((11, 12), (first, second), ys):
        ref = OB.block_forward(first[0], *inp[1:], heads=heads, window=w, shift=s, m=m,
                               dtype=dtype, round_output=False)
        check(y, ref, dtype, f"block with the weights of seed {seed}",
              beyond_bar=BLOCK_BEYOND_BF16)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("C,heads,w,s,m", [(32, 1, 8, 4, 8), (96, 3, 8, 4, 16), (180, 6, 16, 8, 32),
                                             (256, 8, 8, 4, 16)])
def test_block_prepacked_weights(dtype, C, heads, w, s, m):
    """nystra_block_forward_packed on an image packed once gives, bit for bit,
    what nystra_block_forward gives with its per-call packing, on two inputs
    in a row (one image, one workspace)."""
    inp = W.block_inputs(1, 32, 32, C, seed=21, dtype=dtype)
    other = W.block_inputs(1, 32, 32, C, seed=22, dtype=dtype)[0]
    wq, bq, wp, bp = (to_dev(a, dtype) for a in inp[1:])
    packed = B.nystra_block_pack_weights(wq, wp)
    assert packed is not None and packed.numel() == B.nystra_block_packed_size(
        C, B.F32 if dtype == "f32" else B.BF16)
    for xh in (inp[0], other):
        x = to_dev(xh, dtype)
        y0 = B.nystra_block_forward(x, wq, bq, wp, bp, heads, w, shift=s, m=m)
        y1 = B.nystra_block_forward(x, wq, bq, wp, bp, heads, w, shift=s, m=m, packed=packed)
        torch.cuda.synchronize()
        assert torch.equal(y0, y1)
    ref = OB.block_forward(other, *inp[1:], heads=heads, window=w, shift=s, m=m, dtype=dtype,
                           round_output=False)
    check(to_host(y1), ref, dtype, "prepacked block", beyond_bar=BLOCK_BEYOND_BF16)


def test_block_prepacked_not_needed_past_256_channels():
    """Past 256 channels there is no image: packing is a no-op and the packed
    forward takes a NULL image."""
    C, heads = 288, 4
    inp = W.block_inputs(1, 16, 16, C, seed=23, dtype="f32")
    x, wq, bq, wp, bp = (to_dev(a, "f32") for a in inp)
    assert B.nystra_block_packed_size(C) == 0
    assert B.nystra_block_pack_weights(wq, wp) is None
    y0 = B.nystra_block_forward(x, wq, bq, wp, bp, heads, 8, shift=4, m=16)
    y1 = torch.empty_like(y0)
    shape = B.BlockShape(1, 16, 16, C, heads, 8, 4)
    need = B.nystra_block_workspace_size(shape, 16)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    rc = B.lib().nystra_block_forward_packed(
        x.data_ptr(), wq.data_ptr(), bq.data_ptr(), wp.data_ptr(), bp.data_ptr(), None, 0,
        y1.data_ptr(), B.ctypes.byref(shape), 16, B.F32, None, B.BLOCK_NYSTROM, ws.data_ptr(),
        need, None)
    assert rc == 0
    torch.cuda.synchronize()
    assert torch.equal(y0, y1)
