"""ctypes front end of the float64 C oracle (``nystra_oracle.c``).

Test infrastructure: arrays go in and out as float64 numpy arrays; nothing
here touches a GPU.  Each wrapper names the step of the paper it follows.
"""
import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libnystra_oracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_geometry.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _ip]
    lib.oracle_landmark_map.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _ip]
    lib.oracle_pinv.argtypes = [_dp, _dp, ctypes.c_int, ctypes.c_int]
    lib.oracle_unit_trace.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_double] + [_dp] * 11
    lib.oracle_forward.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_long, ctypes.c_int,
                                   ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                   ctypes.c_double, ctypes.c_int, _dp]
    lib.oracle_exact.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_long, ctypes.c_int,
                                 ctypes.c_int, ctypes.c_double, ctypes.c_int]
    lib.oracle_max_threads.argtypes = []
    for f in (lib.oracle_geometry, lib.oracle_landmark_map, lib.oracle_pinv,
              lib.oracle_unit_trace, lib.oracle_forward, lib.oracle_exact,
              lib.oracle_max_threads):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(_dp)


def _f64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with status {rc}")


def default_scale(d):
    """Per-head softmax scale 1/sqrt(d_h) (Eq. (1), applied per head)."""
    return 1.0 / math.sqrt(d)


def max_threads():
    return _load().oracle_max_threads()


def geometry(N, m, mode=0):
    """(rows, cols, patch_rows, patch_cols, grid_cols) of the pooling grid."""
    out = (ctypes.c_int32 * 5)()
    _check(_load().oracle_geometry(N, m, mode, out), "geometry")
    return tuple(int(v) for v in out)


def landmark_map(N, m, mode=0):
    """int32[N]: landmark index of every token (Step 1, Sec. 2.2 pooling)."""
    out = np.zeros(N, dtype=np.int32)
    _check(_load().oracle_landmark_map(N, m, mode, out.ctypes.data_as(_ip)), "landmark_map")
    return out


def pinv(A, iters):
    """Step 4: iterative pseudo-inverse of a square matrix A."""
    A = _f64(A)
    m = A.shape[0]
    Z = np.zeros((m, m), dtype=np.float64)
    _check(_load().oracle_pinv(_ptr(A), _ptr(Z), m, iters), "pinv")
    return Z


def unit_trace(Q, K, V, m, iters=6, mode=0, scale=None):
    """One unit with all intermediates of Algorithm 1 / Eq. (8)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    N, d = Q.shape
    if scale is None:
        scale = default_scale(d)
    out = {
        "O": np.zeros((N, d)), "Qbar": np.zeros((m, d)), "Kbar": np.zeros((m, d)),
        "mL": np.zeros(N), "mU": np.zeros(m), "GL": np.zeros((N, m)),
        "GU": np.zeros((m, N)), "GA": np.zeros((m, m)), "Z": np.zeros((m, m)),
        "P": np.zeros((N, m)), "ON": np.zeros((N, d)), "OD": np.zeros(N),
    }
    names = ["Qbar", "Kbar", "mL", "mU", "GL", "GU", "GA", "Z", "P", "ON", "OD"]
    rc = _load().oracle_unit_trace(_ptr(Q), _ptr(K), _ptr(V), _ptr(out["O"]), N, d, m, iters,
                                   mode, float(scale), *[_ptr(out[n]) for n in names])
    _check(rc, "unit_trace")
    return out


def forward(Q, K, V, m, iters=6, mode=0, scale=None, n_threads=0, diag=False):
    """Batched PnP-Nystra over [..., N, d] inputs (all leading dims are units).

    With diag, also returns per unit (units x 3): min O_D, max O_D (Step 7's
    denominators) and ||I - G_A^n Z_K||_F (the Step 4 residual)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    shape = Q.shape
    N, d = shape[-2], shape[-1]
    units = int(np.prod(shape[:-2])) if len(shape) > 2 else 1
    if scale is None:
        scale = default_scale(d)
    O = np.zeros(shape, dtype=np.float64)
    dg = np.zeros((units, 3), dtype=np.float64) if diag else None
    rc = _load().oracle_forward(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), units, N, d, m, iters,
                                mode, float(scale), int(n_threads), _ptr(dg))
    _check(rc, "forward")
    return (O, dg) if diag else O


def exact(Q, K, V, scale=None, n_threads=0):
    """Batched exact softmax attention, Eq. (1), over [..., N, d] inputs."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    shape = Q.shape
    N, d = shape[-2], shape[-1]
    units = int(np.prod(shape[:-2])) if len(shape) > 2 else 1
    if scale is None:
        scale = default_scale(d)
    O = np.zeros(shape, dtype=np.float64)
    rc = _load().oracle_exact(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), units, N, d, float(scale),
                              int(n_threads))
    _check(rc, "exact")
    return O
