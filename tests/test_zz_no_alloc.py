"""The allocation-free entry point (nystra_attn_forward_noalloc) through the C
ABI, against the workspace entry point it mirrors (nystra_attn_forward_ws,
which runs the same kernels on a torch-allocated workspace): bit-identical
outputs on consecutive calls, the later ones smaller, each also within the
parity bar of the float64 oracle."""
import pytest

import oracle
from paper_2506_08520_amd import binding as B
from paper_2506_08520_amd import workloads as W
from helpers import check, to_dev, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# (n_windows, heads, N, d_h, m, dtype, variant): token-split shapes that use
# the static scratch, each smaller than the one before, then a 64-token shape
# whose kernel needs no scratch at all.
CALLS = [(1, 3, 65536, 32, 64, "f32", B.VARIANT_AUTO),
         (1, 2, 16384, 30, 32, "bf16", B.VARIANT_AUTO),
         (2, 2, 1024, 32, 16, "f32", B.VARIANT_SPLIT),
         (4, 6, 64, 30, 16, "f32", B.VARIANT_AUTO)]


def test_noalloc_matches_workspace_entry():
    for nw, h, N, d, m, dtype, variant in CALLS:
        code = B.F32 if dtype == "f32" else B.BF16
        opts = B.make_opts(variant=variant)
        need = B.nystra_attn_workspace_size(nw, h, N, d, m, code, opts)
        assert need <= B.STATIC_SCRATCH_BYTES
        assert (need > 0) == (N > 64)
        q, k, v = W.iid((nw, h, N, d), seed=N + d + m, dtype=dtype)
        tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
        ref = B.nystra_attn_forward_ws(tq, tk, tv, m, opts=opts)
        got = B.nystra_attn_forward_noalloc(tq, tk, tv, m, opts=opts)
        torch.cuda.synchronize()
        what = f"noalloc {(nw, h, N, d, m, dtype)} workspace {need} B"
        print(what, flush=True)
        assert torch.equal(got, ref), what
        check(to_host(got), oracle.forward(q, k, v, m), dtype, what)
