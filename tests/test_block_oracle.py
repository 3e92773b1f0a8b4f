"""Pins of the float64 block oracle (window partition, projections, head
split and merge, window reverse) against facts it does not compute itself."""
import numpy as np
import pytest

from oracle import block as OB

torch = pytest.importorskip("torch")


def weights(C, seed):
    rng = np.random.default_rng(seed)
    return (rng.normal(0, C ** -0.5, (C, 3 * C)), rng.normal(0, 0.1, 3 * C),
            rng.normal(0, C ** -0.5, (C, C)), rng.normal(0, 0.1, C))


@pytest.mark.parametrize("B,H,W,w,s", [(1, 8, 8, 4, 0), (2, 8, 12, 4, 2), (1, 16, 8, 8, 4),
                                       (3, 6, 6, 3, 1), (1, 4, 4, 4, 3)])
def test_partition_two_formulations(B, H, W, w, s):
    a = OB.window_tokens_loops(B, H, W, w, s)
    b = OB.window_tokens_roll(B, H, W, w, s)
    assert np.array_equal(a, b)
    assert np.array_equal(np.sort(a.reshape(-1)), np.arange(B * H * W))   # a permutation


def brute_global_block(x, wq, bq, wp, bp, heads):
    """Global softmax attention over every pixel of one image, written out
    directly: no window table, no oracle attention."""
    H, W, C = x.shape[1:]
    d = C // heads
    t = x.reshape(H * W, C)
    qkv = t @ wq + bq
    out = np.zeros((H * W, C))
    for h in range(heads):
        q = qkv[:, h * d:(h + 1) * d]
        k = qkv[:, C + h * d:C + (h + 1) * d]
        v = qkv[:, 2 * C + h * d:2 * C + (h + 1) * d]
        s = q @ k.T / np.sqrt(d)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        out[:, h * d:(h + 1) * d] = (p / p.sum(axis=1, keepdims=True)) @ v
    return (out @ wp + bp).reshape(1, H, W, C)


def test_global_window_equals_brute_force():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(1, 8, 8, 12))
    wq, bq, wp, bp = weights(12, 2)
    got = OB.block_forward(x, wq, bq, wp, bp, heads=3, window=8, attention="exact")
    assert np.abs(got - brute_global_block(x, wq, bq, wp, bp, 3)).max() < 1e-12


@pytest.mark.parametrize("s", [1, 3, 5])
def test_shift_invariance_of_global_exact_attention(s):
    """Attention over all tokens commutes with any permutation of them, so a
    cyclic shift of a whole-map window, undone on the way out, changes
    nothing."""
    rng = np.random.default_rng(3)
    x = rng.normal(size=(2, 8, 8, 8))
    wq, bq, wp, bp = weights(8, 4)
    a = OB.block_forward(x, wq, bq, wp, bp, heads=2, window=8, shift=0, attention="exact")
    b = OB.block_forward(x, wq, bq, wp, bp, heads=2, window=8, shift=s, attention="exact")
    assert np.abs(a - b).max() < 1e-12


@pytest.mark.parametrize("attention", ["nystrom", "exact"])
def test_value_bias_passes_through(attention):
    """Normalised rows (softmax, and Eq. (8)'s division by O_D) make
    O(V + 1 delta^T) = O + 1 delta^T, so adding delta to the value bias adds
    delta W_proj to every output pixel, with every head's slice of delta in
    its own place."""
    rng = np.random.default_rng(5)
    C, heads = 12, 3
    x = rng.normal(size=(1, 8, 8, C))
    wq, bq, wp, bp = weights(C, 6)
    delta = rng.normal(size=C)
    bq2 = bq.copy()
    bq2[2 * C:] += delta
    kw = dict(heads=heads, window=4, shift=2, m=4, attention=attention)
    a = OB.block_forward(x, wq, bq, wp, bp, **kw)
    b = OB.block_forward(x, wq, bq2, wp, bp, **kw)
    assert np.abs((b - a) - delta @ wp).max() < 1e-10


def test_nystrom_with_one_token_per_landmark_is_exact():
    """m = N (every landmark one token): the Nystrom reconstruction of Eq. (8)
    is exact once the pseudo-inverse has converged."""
    rng = np.random.default_rng(7)
    x = rng.normal(size=(1, 8, 8, 8)) * 0.5
    wq, bq, wp, bp = weights(8, 8)
    kw = dict(heads=2, window=4, shift=1)
    a = OB.block_forward(x, wq, bq, wp, bp, m=16, iters=40, attention="nystrom", **kw)
    b = OB.block_forward(x, wq, bq, wp, bp, attention="exact", **kw)
    assert np.abs(a - b).max() < 1e-8


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(9)
    x = np.concatenate([rng.normal(size=4000) * 10.0 ** rng.integers(-5, 5, 4000),
                        [0.0, -0.0, 1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -3.5]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).double().numpy()
    assert np.array_equal(OB.round_bf16(x), ref)
