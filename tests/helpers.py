"""Shared helpers of the GPU parity tests."""
import numpy as np

# Parity bars: fp32 outputs within 1e-4 max-abs of the float64 oracle; bf16
# outputs within 2e-2 of the oracle's output RMS in max-abs.  In bf16 the error
# that is left after allowing every element the half-ulp that rounding the
# exact result to bf16 costs must in addition stay within BEYOND_BF16 of RMS:
# the kernels' own arithmetic error is ~1e-4 of RMS, so a change that lost
# precision inside a kernel (say, a dropped lo term of a split operand) fails
# here even where the storage rounding dominates the literal figure.
TOL = {"f32": 1e-4, "bf16": 2e-2}
BEYOND_BF16 = 2e-3


def torch_dtype(dtype):
    import torch
    return torch.float32 if dtype == "f32" else torch.bfloat16


def to_dev(x, dtype):
    """float64 numpy holding dtype-representable values -> device tensor (exact)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(torch_dtype(dtype)).cuda()


def to_host(t):
    return t.float().cpu().double().numpy()


def bf16_half_ulp(x):
    """Half a bf16 unit in the last place at |x| (the storage rounding floor)."""
    a = np.maximum(np.abs(x), np.finfo(np.float32).tiny)
    return np.exp2(np.floor(np.log2(a)) - 8)


def round_bf16(x):
    """float64 -> nearest fp32 -> nearest-even bf16, returned as float64."""
    u = np.asarray(x, dtype=np.float64).astype(np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def error(got, ref, dtype, storage_floor=False):
    """fp32: max-abs; bf16: max-abs relative to the oracle's output RMS.

    With storage_floor, each bf16 element is first allowed the half-ulp by
    which the kernel's own rounding to bf16 can have moved it: rounding an
    fp32 result o to the stored value got costs at most half an ulp at |got|
    (rounding never leaves o's binade downwards, and upwards only to the
    power of two that starts the next one), so what remains is a lower bound
    on the arithmetic error before the store.
    """
    if not got.size:
        return 0.0
    diff = np.abs(got - ref)
    if dtype == "f32":
        return float(diff.max())
    if storage_floor:
        diff = np.maximum(diff - bf16_half_ulp(got), 0.0)
    rms = float(np.sqrt((ref ** 2).mean()))
    return float(diff.max()) / rms


def check(got, ref, dtype, what, beyond_bar=BEYOND_BF16, allowance=None):
    """The parity bar, printed and asserted.

    fp32: max-abs <= 1e-4.  bf16: the error beyond the storage rounding
    <= beyond_bar x RMS, and the literal max-abs <= 2e-2 x RMS wherever the
    oracle's own output, rounded to bf16, meets that literal bar (a kernel
    without any arithmetic error could not do better than that rounding; on
    heavy-tailed outputs, max|O| >> RMS, it alone exceeds 2e-2) -- with an
    allowance, wherever that rounding plus the largest allowance meets it.
    `allowance` (bf16 only) is a per-element bound on an error the kernel
    makes by design, taken off before the beyond-rounding bar (the exact
    kernel's bf16 probabilities).  Returns the figures."""
    assert got.shape == ref.shape
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    if dtype == "f32":
        err = error(got, ref, dtype)
        print(f"{what}: max-abs {err:.3e}")
        assert err <= TOL[dtype], f"{what}: max-abs {err:.3e}"
        return {"max_abs": err}
    lit = error(got, ref, dtype)
    beyond = error(got, ref, dtype, storage_floor=True)
    rms = float(np.sqrt((ref ** 2).mean())) if ref.size else 1.0
    floor = float(np.abs(round_bf16(ref) - ref).max()) / rms if ref.size else 0.0
    msg = (f"{what}: max-abs/RMS {lit:.3e} (bf16 rounding of the oracle alone {floor:.3e}), "
           f"beyond bf16 rounding {beyond:.3e}")
    attainable = floor   # what the literal figure can be for a kernel meeting the design
    if allowance is not None:
        rest = np.abs(got - ref) - bf16_half_ulp(got) - allowance
        beyond = float(np.maximum(rest, 0.0).max()) / rms if ref.size else 0.0
        attainable += float(np.max(allowance)) / rms if ref.size else 0.0
        msg += f", beyond rounding and allowance {beyond:.3e}"
    print(msg)
    assert beyond <= beyond_bar, f"{what}: beyond-rounding error {beyond:.3e} > {beyond_bar}"
    if attainable <= TOL[dtype]:
        assert lit <= TOL[dtype], f"{what}: max-abs/RMS {lit:.3e}"
    return {"literal": lit, "beyond": beyond, "rounding_floor": floor}


def exact_bf16_allowance(q, k, v, exact):
    """Per-element bound on what the exact kernel's bf16 probabilities cost.

    The bf16 exact kernel sums each row's softmax denominator l in fp32 but
    rounds the probabilities p_ij (in [0, 1]) to bf16 before the P V product,
    as bf16 flash attention does.  Rounding to nearest moves p by at most
    2^-8 p, so output element (i, c) moves by at most
    2^-8 sum_j p_ij |v_jc| / l_i = 2^-8 (softmax(s Q K^T) |V|)_ic: exact
    attention on |V|, from the oracle (`exact` is oracle.exact)."""
    return 2.0 ** -8 * exact(q, k, np.abs(v))


def sample_units(units, count):
    """Deterministic strided subset of unit indices, first and last included."""
    if count is None or units <= count:
        return np.arange(units)
    idx = np.unique(np.linspace(0, units - 1, count).round().astype(np.int64))
    return idx
