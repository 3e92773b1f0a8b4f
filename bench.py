"""Benchmark of the PnP-Nystra window-attention hot path on one MI355X.

One step = one PnP-Nystra forward (landmark pooling, kernel blocks,
pseudo-inverse, value products, normalisation -- the whole path, one fused
launch) over the SwinIR-like layer: a 256x256x180 feature map in 8x8 windows,
1024 windows x 6 heads, N = 64, d_h = 30, m = 16 landmarks, K = 6
pseudo-inverse iterations, fp32 storage.  Every other workload (the 8x8,
16x16 and 32x32 window configurations in each storage type they are run in)
is timed the same way and reported in "configs": kernel time, tokens/s, HBM
and matrix-core fractions of the MI355X peaks, and exact attention on the
same buffers with its own distance from its floor.  Inputs are synthetic
(seeded) and resident in HBM; the steps rotate over enough copies of them
(> 1 GiB) that no step is served from the 256 MB Infinity Cache.

Prints ONE JSON line (rank 0, N = 1 GPU).
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E peak, GB/s
# Dense matrix-core peaks by storage type (fp32 inputs run the fp32 matrix
# cores, bf16 inputs the bf16 ones), TFLOP/s.
MFMA_PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
# v_exp_f32 per second: a quarter of the unpacked fp32 lane rate
# (157.3 TFLOP/s = 2 flops x 2 packed lanes x 39.3 T lane-ops/s).
EXP_PEAK_PER_S = 157.3e12 / 4 / 4
ROTATE_BYTES = 1.2 * (1 << 30)  # working set cycled by the timed steps


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--preheat", type=float, default=1.0,
                    help="seconds of untimed launches before the warm-up steps, so the GPU "
                         "runs at its steady clocks (0: none); reported as preheat_s")
    ap.add_argument("--config", default="c2")
    ap.add_argument("--dtype", default="f32", choices=["f32", "bf16"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-exact", action="store_true", help="skip the exact-attention timing")
    ap.add_argument("--no-alt", action="store_true",
                    help="time only the headline workload (--config, --dtype)")
    ap.add_argument("--configs", default=",".join(ALL_CASES),
                    help="config:dtype pairs timed besides the headline, one record each")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the same-traffic elementwise kernel (the practical HBM ceiling)")
    ap.add_argument("--graph", action="store_true",
                    help="time one replay of a HIP graph holding the timed launches instead "
                         "of launches issued one by one (measured slower on the 64-token "
                         "layer: c2 fp32 46.5 us against 43.6)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="wall-clock budget of each CPU-baseline leg (all threads, one thread)")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the benchmark line: time PnP-Nystra and exact attention "
                         "over N x m x K on the smooth-field recipe and report the error "
                         "against exact attention (one JSON line per point)")
    ap.add_argument("--sweep-n", default="64,256,1024,4096")
    ap.add_argument("--sweep-m", default="8,16,32,64")
    ap.add_argument("--sweep-k", default="1,3,4,5,6")
    ap.add_argument("--block", default=None,
                    help="comma-separated block layers to time (swinir, uformer, win16, win32, "
                         "global) or 'all': the window-attention block with PnP-Nystra vs exact")
    ap.add_argument("--sweep-side", type=int, default=512,
                    help="side of the square feature map the sweep cuts into windows")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="also run a plain device-to-device copy of this many MiB (3 times), "
                         "the reference kernel for scaling HBM byte counters")
    return ap.parse_args()


class Case:
    """Device copies of one workload, rotated across steps."""

    def __init__(self, wl, dtype, q, k, v):
        import torch
        from paper_2506_08520_amd import workloads as W  # noqa: F401
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        self.wl, self.dtype = wl, dtype
        self.io_bytes = wl.io_bytes(dtype)
        self.nsets = max(2, math.ceil(ROTATE_BYTES / self.io_bytes))
        base = [torch.from_numpy(x).to(tdt).cuda() for x in (q, k, v)]
        self.sets = []
        for i in range(self.nsets):
            trip = base if i == 0 else [t.clone() for t in base]
            self.sets.append((*trip, torch.empty_like(base[0])))


def time_kernel(case, launch, steps, warmup, preheat=0.0, graph=False):
    """Preheat for `preheat` seconds and run `warmup` untimed launches, then
    time exactly `steps` launches, one per step, back to back.

    The launches are issued one by one on a side stream; with graph they are
    captured once in a HIP graph (stream capture over the rotating buffers)
    and the timed region is one replay of it.

    Returns (ms per step by the host clock between the synchronisations that
    bracket the timed region, ms per launch from one HIP event pair recorded
    on the launch stream around the same region, and -- as a diagnostic only
    -- the 10th, 50th and 90th percentiles of event pairs recorded around
    single eager launches, which include the events' and the host's own
    overhead, and the number of preheat launches)."""
    import torch
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        # The first launches after idle run at lower clocks (c2 fp32: 51.7 us
        # after 20 launches, 46.3 us after a second of them); the preheat runs
        # the same launches for the given time, checked every 64 launches.
        heat, t_end = 0, time.perf_counter() + preheat
        while time.perf_counter() < t_end:
            for _ in range(64):
                launch(*case.sets[heat % case.nsets], stream)
                heat += 1
            stream.synchronize()
        for i in range(warmup):
            launch(*case.sets[i % case.nsets], stream)
        g = None
        if graph:
            stream.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                for i in range(steps):
                    launch(*case.sets[(warmup + i) % case.nsets], stream)
            g.replay()   # untimed: the first replay uploads the graph
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r0.record(stream)
        if graph:
            g.replay()
        else:
            for i in range(steps):
                launch(*case.sets[(warmup + i) % case.nsets], stream)
        r1.record(stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        region = r0.elapsed_time(r1) / steps
        n = min(steps, 50)
        starts = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        stops = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for i in range(n):
            starts[i].record(stream)
            launch(*case.sets[(warmup + steps + i) % case.nsets], stream)
            stops[i].record(stream)
        torch.cuda.synchronize()
    del g
    each = sorted(a.elapsed_time(b) for a, b in zip(starts, stops))
    pct = [each[min(n - 1, int(round(f * (n - 1))))] for f in (0.1, 0.5, 0.9)]
    return (t1 - t0) * 1e3 / steps, region, pct, heat


def measured_traffic(cfg, dtype, variant):
    """HBM bytes per launch from the committed counter record, if the kernel
    it was measured on is still the one in the source tree; else None."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if variant != 2 or not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(f"{cfg}:{dtype}")
    if rec is None:
        return None
    h = hashlib.sha256()
    for f in rec["source_files"]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != rec["source_sha256"]:
        return None
    return rec["fetch_bytes"] + rec["write_bytes"]


def cpu_baseline(wl, q, k, v, budget_s, n_threads=0):
    """The float64 oracle on a bounded sample of the same units: a strided
    subset when the whole workload would overrun the budget, otherwise the
    whole workload repeated until the budget is spent.  n_threads = 0 runs
    OpenMP's default thread count (all cores given to the process)."""
    import numpy as np
    import oracle
    units = wl.units
    flat = [x.reshape(units, wl.N, wl.d) for x in (q, k, v)]
    probe = min(units, 48)
    idx = np.linspace(0, units - 1, probe).round().astype(np.int64)
    t0 = time.perf_counter()
    oracle.forward(*(x[idx] for x in flat), wl.m, n_threads=n_threads)
    t_probe = time.perf_counter() - t0
    per_unit = max(t_probe, 1e-6) / probe
    n = int(min(units, max(probe, budget_s / per_unit)))
    idx = np.linspace(0, units - 1, n).round().astype(np.int64)
    sample = [np.ascontiguousarray(x[idx]) for x in flat]
    passes = []
    t0 = time.perf_counter()
    while True:   # whole passes until the budget is spent (at least one)
        tp = time.perf_counter()
        oracle.forward(*sample, wl.m, n_threads=n_threads)
        passes.append(time.perf_counter() - tp)
        dt = time.perf_counter() - t0
        if dt >= budget_s or n < units:
            break
    reps = len(passes)
    tokens = reps * n * wl.N / wl.heads   # spatial tokens (all heads) processed
    what = (f"all {units} units x {reps} passes" if n == units
            else f"{n} of {units} units, strided")
    cores = oracle.max_threads() if n_threads <= 0 else n_threads
    ps = sorted(passes)
    pct = [ps[min(reps - 1, int(round(f * (reps - 1))))] for f in (0.1, 0.5, 0.9)]
    return {"value": tokens / dt, "unit": "tokens/s", "cores": cores,
            "kind": "oracle", "pass_s_p10_p50_p90": pct,
            "sample": f"{what} of {wl.name} ({wl.N} tokens, m={wl.m}, K=6); float64 C "
                      f"oracle, {cores} thread(s), {dt:.1f} s wall"}


def sweep(args):
    """(m, K, N) sweep on the c4-style smooth field: a side x side x 180 map
    (6 heads, d_h = 30; side 512 by default) cut into windows of N tokens, so
    the number of units falls as N grows (24576 units at N = 64 ... 6 at
    N = 262144, one window per map).  Per point: kernel times (one event pair
    around back-to-back launches on the same buffers) of the one-pass kernels
    (nystra_attn_forward_ex), of the token-split kernels (forced, through
    nystra_attn_forward_ws, where they cover the shape), of the automatic
    choice of nystra_attn_forward_ws and of exact attention, and the error of
    that choice against exact attention over all outputs."""
    import torch
    from paper_2506_08520_amd import binding as B
    from paper_2506_08520_amd import workloads as W

    B.lib()
    base = W.CONFIGS["c4"]
    side, heads, d = args.sweep_side, base.heads, base.d

    def timed(fn, reps):
        s = torch.cuda.current_stream()
        fn()
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        r0.record(s)
        for _ in range(reps):
            fn()
        r1.record(s)
        torch.cuda.synchronize()
        return r0.elapsed_time(r1) / reps

    names = {B.VARIANT_GENERIC: "generic", B.VARIANT_TILED: "mfma-tiled",
             B.VARIANT_SPLIT: "token-split"}
    for N in (int(x) for x in args.sweep_n.split(",")):
        w = int(round(N ** 0.5))
        wl = W.Workload(f"sweep-N{N}", (side // w) ** 2, heads, N, d, base.m, ("f32",), "smooth",
                        base.seed, f"smooth field {side}x{side}x{heads * d}, {w}x{w} windows")
        q, k, v = (torch.from_numpy(x).float().cuda() for x in W.generate(wl, "f32"))
        for dt in (args.dtype,):
            code = B.F32 if dt == "f32" else B.BF16
            tdt = torch.float32 if dt == "f32" else torch.bfloat16
            tq, tk, tv = (x.to(tdt) for x in (q, k, v))
            ex = torch.empty_like(tq)
            reps = max(3, min(50, int(2e5 // (wl.units * N / 64))))
            t_ex = exf = None
            if not args.no_exact:
                t_ex = timed(lambda: B.nystra_exact_attn_forward(tq, tk, tv, out=ex), reps)
                exf = ex.float()
                ref_rms = float(exf.pow(2).mean().sqrt())
            for m in (int(x) for x in args.sweep_m.split(",")):
                if m > N:
                    continue
                for K in (int(x) for x in args.sweep_k.split(",")):
                    o = torch.empty_like(tq)
                    opts = B.make_opts(pinv_iters=K)
                    t1 = timed(lambda: B.nystra_attn_forward_ex(tq, tk, tv, m, opts=opts, out=o),
                               reps)
                    sopts = B.make_opts(pinv_iters=K, variant=B.VARIANT_SPLIT)
                    t_split = None
                    try:
                        nb = B.nystra_attn_workspace_size(wl.n_windows, heads, N, d, m, code,
                                                          sopts)
                    except B.NystraError:
                        nb = 0
                    if nb:
                        wsb = torch.empty(nb, dtype=torch.uint8, device="cuda")
                        t_split = timed(lambda: B.nystra_attn_forward_ws(
                            tq, tk, tv, m, opts=sopts, workspace=wsb, out=o), reps)
                        del wsb
                    na = B.nystra_attn_workspace_size(wl.n_windows, heads, N, d, m, code, opts)
                    wsa = torch.empty(max(na, 1), dtype=torch.uint8, device="cuda")
                    t = timed(lambda: B.nystra_attn_forward_ws(tq, tk, tv, m, opts=opts,
                                                               workspace=wsa, out=o), reps)
                    diff = (o.float() - exf) if exf is not None else None
                    one = names[B.nystra_select_variant(N, d, m, code, opts)]
                    print(json.dumps({
                        "N": N, "m": m, "K": K, "dtype": dt, "units": wl.units,
                        "variant": "token-split" if na else one,
                        "nystra_us": round(t * 1e3, 2), "onepass_variant": one,
                        "onepass_us": round(t1 * 1e3, 2),
                        "split_us": round(t_split * 1e3, 2) if t_split else None,
                        "exact_us": round(t_ex * 1e3, 2) if t_ex else None,
                        "speedup_vs_exact": round(t_ex / t, 3) if t_ex else None,
                        "rel_rms_err_vs_exact":
                            float(diff.pow(2).mean().sqrt()) / ref_rms if t_ex else None,
                        "max_abs_err_vs_exact": float(diff.abs().max()) if t_ex else None}),
                          flush=True)
                    del wsa
        del q, k, v, tq, tk, tv, ex
        torch.cuda.empty_cache()
    return 0


# Window-attention block layers (the c2-c5 layers as whole blocks, and one
# global window): (map side, channels, heads, window, m).
BLOCK_LAYERS = {
    "swinir": (256, 180, 6, 8, 16),    # c2: 8x8 windows, 6 heads of 30
    "uformer": (512, 32, 1, 8, 8),     # c3: 8x8 windows, 1 head of 32
    "win16": (512, 180, 6, 16, 32),    # c4: 16x16 windows
    "win32": (512, 256, 8, 32, 64),    # c5: 32x32 windows, 8 heads of 32
    "global": (512, 180, 6, 512, 64),  # one window per map
}


def block_bench(args):
    """Per layer: one block call (QKV projection with window partition and a
    shift of half a window, attention, head merge, output projection, window
    reverse) with PnP-Nystra and with exact attention, the attention operator
    alone on the same Q, K, V, and the projections' achieved rate."""
    import torch
    from paper_2506_08520_amd import binding as B
    from paper_2506_08520_amd import workloads as W

    B.lib()
    names = list(BLOCK_LAYERS) if args.block == "all" else args.block.split(",")

    def timed(fn, reps):
        s = torch.cuda.current_stream()
        for _ in range(max(3, reps // 2)):   # warm-up: clocks, caches, first-call costs
            fn()
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        r0.record(s)
        for _ in range(reps):
            fn()
        r1.record(s)
        torch.cuda.synchronize()
        return r0.elapsed_time(r1) / reps * 1e3   # us

    for name in names:
        side, C, heads, w, m = BLOCK_LAYERS[name]
        shift = w // 2 if w < side else 0
        dt = args.dtype
        tdt = torch.float32 if dt == "f32" else torch.bfloat16
        x, wq, bq, wp, bp = (torch.from_numpy(a).to(tdt).cuda()
                             for a in W.block_inputs(1, side, side, C, seed=4242, dtype=dt))
        code = B.F32 if dt == "f32" else B.BF16
        shape = B.BlockShape(1, side, side, C, heads, w, shift)
        y = torch.empty_like(x)
        res = {"layer": name, "dtype": dt, "map": f"{side}x{side}x{C}", "heads": heads,
               "window": w, "shift": shift, "m": m, "tokens": side * side}
        reps = 20 if w < side else 5
        for att, key in ((B.BLOCK_NYSTROM, "nystrom"), (B.BLOCK_EXACT, "exact")):
            if key == "exact" and args.no_exact:
                continue
            nb = B.nystra_block_workspace_size(shape, m, code, None, att)
            ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
            res[f"block_{key}_us"] = round(timed(lambda: B.nystra_block_forward(
                x, wq, bq, wp, bp, heads, w, shift=shift, m=m, attention=att, workspace=ws,
                out=y), reps if key == "nystrom" or w <= 32 else 3), 2)
            if key == "nystrom":
                # the weights packed once, as for inference (no per-call packing)
                packed = B.nystra_block_pack_weights(wq.view(C, 3 * C), wp.view(C, C))
                res["block_nystrom_prepacked_us"] = round(timed(lambda: B.nystra_block_forward(
                    x, wq, bq, wp, bp, heads, w, shift=shift, m=m, attention=att, workspace=ws,
                    out=y, packed=packed), reps), 2)
                del packed
            del ws
        # the attention alone on window-partitioned tensors of the same size
        nw = (side // w) ** 2
        q, k, v = (torch.randn(nw, heads, w * w, C // heads, device="cuda").to(tdt)
                   for _ in range(3))
        o = torch.empty_like(q)
        na = B.nystra_attn_workspace_size(nw, heads, w * w, C // heads, m, code)
        wsa = torch.empty(max(na, 1), dtype=torch.uint8, device="cuda")
        res["attention_nystrom_us"] = round(timed(lambda: B.nystra_attn_forward_ws(
            q, k, v, m, workspace=wsa, out=o), reps), 2)
        if not args.no_exact:
            res["attention_exact_us"] = round(timed(lambda: B.nystra_exact_attn_forward(
                q, k, v, out=o), reps if w <= 32 else 3), 2)
            res["block_speedup_vs_exact"] = round(res["block_exact_us"] / res["block_nystrom_us"], 3)
        # the SwinIR-shaped transformer block (LayerNorm, window attention,
        # residual, LayerNorm, MLP of ratio 2, residual) with each attention
        from paper_2506_08520_amd.module import SwinTransformerBlock
        for key in ("nystrom", "exact"):
            if key == "exact" and (args.no_exact or w == side):
                continue
            torch.manual_seed(7)
            blk = SwinTransformerBlock(C, heads, w, shift, m=m, attention=key, dtype=tdt)
            with torch.no_grad():
                blk.attn.w_qkv.copy_(wq.view(C, 3 * C))
                blk.attn.b_qkv.copy_(bq)
                blk.attn.w_proj.copy_(wp.view(C, C))
                blk.attn.b_proj.copy_(bp)
            res[f"transformer_block_{key}_us"] = round(timed(lambda: blk(x), reps), 2)
            del blk
        if "transformer_block_exact_us" in res:
            res["transformer_block_speedup_vs_exact"] = round(
                res["transformer_block_exact_us"] / res["transformer_block_nystrom_us"], 3)
        proj_us = res["block_nystrom_us"] - res["attention_nystrom_us"]
        flops = 8.0 * side * side * C * C   # 2 rows C 3C + 2 rows C C
        res["projections_us"] = round(proj_us, 2)
        res["projections_tflops"] = round(flops / (proj_us * 1e-6) / 1e12, 1)
        print(json.dumps(res), flush=True)
        del x, wq, bq, wp, bp, y, q, k, v, o, wsa
        torch.cuda.empty_cache()
    return 0


# The measured workloads: every (configuration, storage type) pair.
ALL_CASES = ("c1:f32", "c2:f32", "c2:bf16", "c3:bf16", "c4:f32", "c4:bf16", "c5:bf16")


def nystrom_flops(N, d, m, K):
    """Algorithmic flops of one unit of Algorithm 1 as the kernels evaluate
    it (Steps 5-6 re-associated): Step 1 pooling sums (2 N d), S_L and S_U
    (4 N m d), S_A (2 m^2 d), the pseudo-inverse (8 K m^3: four m x m
    products per iteration), T = G_U^n [V | 1] and [O_N | O_D] = G_L^n W
    (4 N m (d + 1)), W = Z T (2 m^2 (d + 1)) and the division (N d)."""
    return (2 * N * d + 4 * N * m * d + 2 * m * m * d + 8 * K * m ** 3 + 4 * N * m * (d + 1) +
            2 * m * m * (d + 1) + N * d)


def exact_flops(N, d):
    """Exact attention, Eq. (1): S = Q K^T and P V, 4 N^2 d flops per unit."""
    return 4 * N * N * d


def floors(wl, dtype, flops, exps):
    """Lower bounds (ms) of one launch on MI355X: HBM bytes at 8 TB/s, the
    flops at the matrix-core peak of the storage type, the exponentials at
    the transcendental rate."""
    hbm = wl.io_bytes(dtype) / (HBM_PEAK_GBS * 1e9) * 1e3
    mfma = wl.units * flops / (MFMA_PEAK_TFLOPS[dtype] * 1e12) * 1e3
    exp = wl.units * exps / EXP_PEAK_PER_S * 1e3
    return {"hbm": hbm, "mfma": mfma, "exp": exp}


def measure(wl, dtype, args, q, k, v, headline):
    """Times PnP-Nystra (and, unless disabled, exact attention and the
    same-traffic elementwise kernel) on one workload; returns the record."""
    import torch
    from paper_2506_08520_amd import binding as B

    case = Case(wl, dtype, q, k, v)

    def nys(q_, k_, v_, o_, s):
        B.nystra_attn_forward(q_, k_, v_, wl.m, out=o_, stream=s)

    def ex(q_, k_, v_, o_, s):
        B.nystra_exact_attn_forward(q_, k_, v_, out=o_, stream=s)

    steps = args.steps
    ms, kern, pairs, heat = time_kernel(case, nys, steps, args.warmup, args.preheat,
                                        args.graph)
    code = B.F32 if dtype == "f32" else B.BF16
    K = 6
    fl = nystrom_flops(wl.N, wl.d, wl.m, K)
    fl_floor = floors(wl, dtype, fl, 2 * wl.N * wl.m + wl.m * wl.m)
    floor_ms = max(fl_floor["hbm"], fl_floor["mfma"])
    gbs = case.io_bytes / (kern * 1e-3) / 1e9
    tfl = wl.units * fl / (kern * 1e-3) / 1e12
    r = {
        "config": wl.name, "storage": dtype, "n_windows": wl.n_windows, "heads": wl.heads,
        "N": wl.N, "d_h": wl.d, "m": wl.m, "K": K,
        "variant": {B.VARIANT_GENERIC: "generic", B.VARIANT_TILED: "mfma-tiled"}.get(
            B.nystra_select_variant(wl.N, wl.d, wl.m, code), "?"),
        "kernel_ms": kern, "ms_per_step": ms,
        "timing": "one HIP graph replay of the timed launches" if args.graph else "launches issued one by one",
        "eager_launch_ms_p10_p50_p90": [float(x) for x in pairs],
        "tokens_per_s": wl.n_windows * wl.N / (kern * 1e-3),
        "unit_tokens_per_s": wl.units * wl.N / (kern * 1e-3),
        "hbm": {"algorithmic_bytes": case.io_bytes, "achieved_GBs": gbs,
                "frac": gbs / HBM_PEAK_GBS},
        "flops": {"per_unit": fl, "achieved_TFLOPs": tfl,
                  "peak_TFLOPs": MFMA_PEAK_TFLOPS[dtype],
                  "frac": tfl / MFMA_PEAK_TFLOPS[dtype]},
        "bound": "hbm" if fl_floor["hbm"] >= fl_floor["mfma"] else "mfma",
        "floor_ms": floor_ms, "roofline_frac": floor_ms / kern,
        "preheat_launches": heat,
    }
    if not args.no_exact:
        ems, ekern, epairs, _ = time_kernel(case, ex, max(10, steps // 4), args.warmup,
                                            min(args.preheat, 0.3), args.graph)
        ef = floors(wl, dtype, exact_flops(wl.N, wl.d), wl.N * wl.N)
        eb = max(ef, key=ef.get)
        r["exact"] = {"kernel_ms": ekern, "ms_per_step": ems,
                      "eager_launch_ms_p10_p50_p90": [float(x) for x in epairs],
                      "floor_ms": ef[eb], "floor_bound": eb, "floors_ms": ef,
                      "frac_of_floor": ef[eb] / ekern}
        r["speedup_vs_exact"] = ekern / kern
    if not args.no_ceiling and wl.N <= 64:
        # The practical HBM ceiling for this traffic: one elementwise kernel
        # that reads Q, K and V and writes O once (O = Q + K * V), on the
        # same rotating buffers and stream -- the same bytes as one step,
        # with no arithmetic to speak of.
        def same_traffic(q_, k_, v_, o_, s):
            torch.addcmul(q_, k_, v_, out=o_)

        _, ckern, _, _ = time_kernel(case, same_traffic, steps, args.warmup,
                                     min(args.preheat, 0.3), args.graph)
        cg = case.io_bytes / (ckern * 1e-3) / 1e9
        r["same_traffic_ceiling"] = {
            "kernel": "torch.addcmul: reads Q, K, V and writes O once, the bytes of one step",
            "kernel_ms": ckern, "achieved_GBs": cg, "frac": cg / HBM_PEAK_GBS,
            "nystrom_over_ceiling": gbs / cg}
    r["traffic"] = measured_traffic(wl.name, dtype, B.nystra_select_variant(
        wl.N, wl.d, wl.m, code))
    del case
    torch.cuda.empty_cache()
    return r


def host_cpu():
    """CPU model name and the number of cores this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count()
    return model, n


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the method's "
              "(window, head) units are independent, so N GPUs would each run 1/N of the "
              "windows with no communication.", file=sys.stderr)
        return 2
    if args.sweep:
        return sweep(args)
    if args.block:
        return block_bench(args)
    import torch  # noqa: F401
    from paper_2506_08520_amd import binding as B
    from paper_2506_08520_amd import workloads as W

    B.lib()
    head = f"{args.config}:{args.dtype}"
    cases = [head]
    if not args.no_alt:
        cases += [c for c in args.configs.split(",") if c and c != head]
    records = {}
    main_inputs = None
    for cd in cases:
        cfg, dt = cd.split(":")
        wl = W.CONFIGS[cfg]
        q, k, v = W.generate(wl, dt)
        if cd == head:
            main_inputs = (q, k, v)
        records[cd] = measure(wl, dt, args, q, k, v, cd == head)
        print(f"[bench] {cd}: {records[cd]['kernel_ms'] * 1e3:.1f} us"
              + (f", exact {records[cd]['exact']['kernel_ms'] * 1e3:.1f} us"
                 if "exact" in records[cd] else ""), file=sys.stderr, flush=True)
        if cd != head:
            del q, k, v

    r = records[head]
    wl = W.CONFIGS[args.config]
    tokens = wl.n_windows * wl.N
    line = {
        "metric": "Nystrom window-attention tokens/s at 1 MI355X; % peak HBM BW; "
                  "speedup vs exact",
        "value": tokens / (r["ms_per_step"] * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "preheat_s": args.preheat,
        "preheat_launches": r["preheat_launches"],
        "ms_per_step": r["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.description}; {args.dtype} storage, "
                               "K=6 pseudo-inverse iterations, 2-D pooled landmarks",
                   "n_windows": wl.n_windows, "heads": wl.heads, "N": wl.N, "d_h": wl.d,
                   "m": wl.m, "storage": args.dtype},
    }
    if r["bound"] == "hbm":
        line["roofline"] = {"bound": "hbm", "achieved": r["hbm"]["achieved_GBs"],
                            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": r["hbm"]["frac"],
                            "traffic": r["traffic"],
                            "algorithmic_bytes": r["hbm"]["algorithmic_bytes"]}
    else:
        line["roofline"] = {"bound": "mfma", "achieved": r["flops"]["achieved_TFLOPs"],
                            "peak": r["flops"]["peak_TFLOPs"], "unit": "TFLOP/s",
                            "frac": r["flops"]["frac"], "traffic": r["traffic"],
                            "algorithmic_flops": r["flops"]["per_unit"] * wl.units}
    if "speedup_vs_exact" in r:
        line["speedup_vs_exact"] = r["speedup_vs_exact"]
    if "same_traffic_ceiling" in r:
        line["same_traffic_ceiling"] = r["same_traffic_ceiling"]
    line["kernel_ms"] = r["kernel_ms"]
    line["variant"] = r["variant"]
    line["peaks"] = {"hbm_GBs": HBM_PEAK_GBS, "mfma_TFLOPs": MFMA_PEAK_TFLOPS,
                     "exp_per_s": EXP_PEAK_PER_S}
    line["configs"] = records
    if args.copy_mib > 0:
        n = args.copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        line["copy_calibration_bytes"] = 2 * n * 4
    if not args.no_cpu:
        model, ncores = host_cpu()
        cb = cpu_baseline(wl, *main_inputs, args.cpu_seconds, 0)
        one = cpu_baseline(wl, *main_inputs, args.cpu_seconds, 1)
        cb["host_cpu"] = model
        cb["host_cores_available"] = ncores
        cb["single_thread"] = {k_: one[k_] for k_ in ("value", "unit", "cores", "sample",
                                                      "pass_s_p10_p50_p90")}
        line["cpu_baseline"] = cb
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
