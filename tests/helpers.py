"""Shared helpers of the GPU parity tests."""
import numpy as np

# Parity bars: fp32 outputs within 1e-4 max-abs of the float64 oracle; bf16
# outputs within 2e-2 of the oracle's output RMS in max-abs.
TOL = {"f32": 1e-4, "bf16": 2e-2}


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


def error(got, ref, dtype, storage_floor=False):
    """fp32: max-abs; bf16: max-abs relative to the oracle's output RMS.

    With storage_floor, each bf16 element is first allowed the half-ulp by
    which rounding the exact result to bf16 can move it; used for shapes
    whose outputs have max|O| >> RMS(O), where storage rounding alone would
    exceed a bar stated relative to the RMS.
    """
    if not got.size:
        return 0.0
    diff = np.abs(got - ref)
    if dtype == "f32":
        return float(diff.max())
    if storage_floor:
        diff = np.maximum(diff - bf16_half_ulp(ref), 0.0)
    rms = float(np.sqrt((ref ** 2).mean()))
    return float(diff.max()) / rms


def sample_units(units, count):
    """Deterministic strided subset of unit indices, first and last included."""
    if units <= count:
        return np.arange(units)
    idx = np.unique(np.linspace(0, units - 1, count).round().astype(np.int64))
    return idx
