"""Benchmark of the GPTQ-2D hot path on one MI355X.

One step = one pass of the whole path over one synthetic problem: the
factorisation of both bases (Gram, Cholesky, triangular inverse,
normalisation) followed by the rounding sweep with the objective, all through
the C ABI, with inputs already resident in device memory. The default
workload is 4096 x 4096 with fp32 inputs (X = LLM-like weights in step units,
bases from Student-t(4) activation Grams), computed in fp64.

Prints one JSON line: rounded entries/s over the timed steps, the roofline of
the dominant kernel (the sweep's stage kernel, fp64 MFMA bound), and the CPU
oracle timed on a bounded sample on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "rounded entries/s at 4096×4096 fp32 + % of HBM/MFMA roofline"
PEAK_F64_TFLOPS = 78.6     # MI355X dense fp64 (MFMA and vector)
PEAK_F32_TFLOPS = 157.3    # MI355X dense fp32 (reference only: the path accumulates in fp64)
PEAK_HBM_GBS = 8000.0

WORKLOADS = {
    1: "64x64 fp64 inputs, X=4N(0,1), Wishart(256) bases",
    2: "512x384 fp32 inputs, X=3N(0,1), anisotropic Wishart(2048) bases",
    3: "4096x4096 fp32 inputs, X=N(0,0.02^2)/(0.02/3), Student-t(4) activation-Gram bases (8192 rows)",
    4: "4096x11008 fp32 inputs, X=3N(0,1), spiked-covariance activation-Gram bases (16384 rows)",
    5: "8192x8192 inputs, X=U[-7.5,7.5], upper-triangular bases",
}


# sources of the stage kernel: the HBM traffic taken from rocprofv3 counters
# is reported only while these are unchanged since the counters were read
STAGE_SOURCES = ("paper_2607_27042_amd/csrc/sweep.hip", "paper_2607_27042_amd/csrc/device.hpp",
                 "paper_2607_27042_amd/csrc/internal.hpp", "paper_2607_27042_amd/build.py")


def stage_sources_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in STAGE_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def stage_traffic(config: int, dtype: str):
    """HBM bytes per stage launch from the committed counter summary of this
    workload (FETCH_SIZE + WRITE_SIZE, copy-calibrated), or None when there is
    none or the stage kernel changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_k_stage_c{config}_{dtype}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as fh:
        for line in fh:
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].split(": ", 1)
                fields[k.strip()] = v.strip().strip("`")
    if fields.get("sources_sha256") != stage_sources_digest():
        return None
    try:
        return float(fields["bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(mib: int):
    """A plain device copy of mib MiB, three times: under rocprofv3 --pmc its
    FETCH_SIZE / WRITE_SIZE per dispatch calibrate the counters against known
    bytes."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def gram_flop(M, side: int, reverse: bool) -> tuple:
    """Flops of the Gram of one side as the library forms it (lower 128 x 128
    tiles, whole diagonal tiles), dense and on the envelope of its panel (the product of two 128-row blocks runs over the
    64-column blocks where both hold a nonzero entry: the rest are exact
    zeros). The panel S has S[p][k] = A[k][d-1-p] (side 0) or B[d-1-p][k]
    (side 1), without the reversal in reverse order. Sides whose dimension is
    not a multiple of 128 are formed densely."""
    import numpy as np
    d = M.shape[0]
    dense = float(d) ** 3  # the lower half of d^3 multiply-adds
    if d % 128:
        return dense, dense
    if side == 0:
        S = M.T if reverse else M[:, ::-1].T
    else:
        S = M if reverse else M[::-1, :]
    nb, nk = d // 128, d // 64
    nz = (S != 0).reshape(nb, 128, nk, 64).any(axis=(1, 3))
    has = nz.any(axis=1)
    lo = np.where(has, nz.argmax(axis=1), nk)
    hi = np.where(has, nk - nz[:, ::-1].argmax(axis=1), 0)
    tile = 2.0 * 128 * 128 * 64  # one 64-deep block of a 128 x 128 tile
    dense_t = env_t = 0.0
    for bp in range(nb):
        w = np.maximum(0, np.minimum(hi[bp], hi[: bp + 1]) - np.maximum(lo[bp], lo[: bp + 1]))
        env_t += tile * float(w.sum())
        dense_t += tile * nk * (bp + 1)
    return dense_t, env_t


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(prob, sample: int, reverse: bool = False, cols: int = 512):
    """The oracle as it stands (explicit-inverse + LDL factors, Algorithm 5
    sweep; in reverse order the same on the index-reversed block), timed on a
    bounded sample of the workload and scaled by the flop count to the full
    problem: the factors of the leading sample x sample block, and the sweep of
    that block's first `cols` columns (an error reaches only later columns, so
    these are the block's own first columns; the block's factors stay out of
    the CPU caches, as the full problem's would)."""
    import numpy as np

    import oracle

    X, A, B = prob.widened()
    s_m, s_n = min(sample, prob.m), min(sample, prob.n)
    k = min(cols, s_n)
    Xs, As, Bs = np.ascontiguousarray(X[:s_m, :s_n]), A[:s_m, :s_m], B[:s_n, :s_n]
    if reverse:
        Xs, As, Bs = oracle.reverse_problem(Xs, As, Bs)
    t0 = time.perf_counter()
    L, lamL, U, lamU = oracle.factors(As, Bs)
    t1 = time.perf_counter()
    if k == s_n:
        oracle.round_nested(Xs, L, U)
    else:
        oracle.round_nested_columns(Xs, L, U, k)
    t2 = time.perf_counter()
    tf, tr = t1 - t0, t2 - t1
    m, n = prob.m, prob.n

    def sweep_madds(rows, ncol, upto):
        # Algorithm 5, column j: the column's own sweep (rows (rows + 1) / 2
        # multiply-adds) and the rank-one push of its errors (rows (ncol - j))
        return upto * rows * (rows + 1) / 2 + rows * (upto * ncol - upto * (upto - 1) / 2)

    scale_f = (m ** 3 + n ** 3) / (s_m ** 3 + s_n ** 3)
    scale_r = sweep_madds(m, n, n) / sweep_madds(s_m, s_n, k)
    t_full = tf * scale_f + tr * scale_r
    swept = f"its first {k} columns" if k < s_n else "all of it"
    return {
        "value": m * n / t_full,
        "unit": "entries/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": (f"leading {s_m}x{s_n} block: factors {tf:.2f} s (explicit inverse + LDL), "
                   f"Algorithm 5 sweep of {swept} {tr:.2f} s; scaled by flop count ((m^3+n^3) and "
                   f"Algorithm 5's multiply-adds) to {m}x{n}"),
        "sample_seconds": tf + tr,
        "cpu_model": _cpu_model(),
    }


def array_baseline_run(prob, sample: int, w: int, dev):
    """The paper's own array-framework realisation of the sweep (Algorithm 4 in
    PyTorch, array_baseline.py), on its padded skew layout (Sec. 5) and on the
    natural layout, timed on the GPU on the leading sample x sample block, next
    to the HIP sweep on the same block; all use the library's factors of that
    block. Scaled to the workload by mn(m+n)."""
    import numpy as np
    import torch

    import array_baseline as ab
    from paper_2607_27042_amd import binding

    s_m, s_n = min(sample, prob.m), min(sample, prob.n)
    X = torch.from_numpy(np.ascontiguousarray(prob.X[:s_m, :s_n])).to(dev)
    A = torch.from_numpy(np.ascontiguousarray(prob.A[:s_m, :s_m])).to(dev)
    B = torch.from_numpy(np.ascontiguousarray(prob.B[:s_n, :s_n])).to(dev)
    f = binding.Factors.from_bases(A, B)
    L, U, _, _ = f.export()
    ws = f.workspace()
    Zh = torch.empty((s_m, s_n), dtype=torch.int32, device=dev)
    Yh = torch.empty_like(X)
    obj = torch.empty(1, dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()
    binding.gptq2d_round(f.handle, X, Zh, Yh, obj, ws, stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(5):
        binding.gptq2d_round(f.handle, X, Zh, Yh, obj, ws, stream)
    torch.cuda.synchronize()
    t_hip = (time.perf_counter() - t0) / 5
    X64 = X.double()
    ab.blocked_sweep(X64[:64, :64].contiguous(), L[:64, :64].contiguous(), U[:64, :64].contiguous(), w=w)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    Za, _, _ = ab.blocked_sweep(X64, L, U, w=w)
    torch.cuda.synchronize()
    t_arr = time.perf_counter() - t0
    mism = int((Za.to(torch.int32) != Zh).sum())
    # the same algorithm on the padded skew layout of Sec. 5
    ab.blocked_sweep_skew(X64[:64, :64].contiguous(), L[:64, :64].contiguous(), U[:64, :64].contiguous(), w=w)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    Zs, _, _ = ab.blocked_sweep_skew(X64, L, U, w=w)
    torch.cuda.synchronize()
    t_skew = time.perf_counter() - t0
    mism_skew = int((Zs.to(torch.int32) != Zh).sum())
    # the implicit-Y form of Appendix B (Algorithm 6), one buffer C = L E
    ab.implicit_sweep(X64[:64, :64].contiguous(), L[:64, :64].contiguous(), U[:64, :64].contiguous())
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    Zi, _, _ = ab.implicit_sweep(X64, L, U)
    torch.cuda.synchronize()
    t_impl = time.perf_counter() - t0
    mism_impl = int((Zi.to(torch.int32) != Zh).sum())
    f.close()
    m, n = prob.m, prob.n
    scale = (m * n * (m + n)) / (s_m * s_n * (s_m + s_n))
    return {
        "value": m * n / (t_skew * scale),
        "unit": "entries/s",
        "kind": "paper Algorithm 4 (blocked, band flushes as windowed batched mat-vecs) on the padded skew "
                "layout of Sec. 5, in PyTorch fp64 on the GPU",
        "sample": f"leading {s_m}x{s_n} block, block width {w}, the library's factors of that block; "
                  f"scaled by mn(m+n) to {m}x{n}",
        "sweep_s": t_skew,
        "hip_sweep_s_same_sample": t_hip,
        "hip_speedup": t_skew / t_hip,
        "z_mismatches_vs_hip": mism_skew,
        "natural_layout_sweep_s": t_arr,
        "natural_layout_z_mismatches_vs_hip": mism,
        "implicit_y_sweep_s": t_impl,
        "implicit_y_z_mismatches_vs_hip": mism_impl,
    }


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_batch(args, dev):
    """A step = gptq2d_factor_batched + gptq2d_round_batched over N problems
    drawn from the config's recipe (layer seeds 0 .. N-1), inputs resident in
    HBM. Prints one JSON line; value = N m n / step time."""
    import torch

    from paper_2607_27042_amd import binding, workloads as wl

    N = args.batch
    log(f"generating {N} problems of config {args.config}")
    probs = [wl.make_config(args.config, args.dtype, layer=i) for i in range(N)]
    m, n = probs[0].m, probs[0].n
    Xs = [torch.from_numpy(p.X).to(dev) for p in probs]
    As = [torch.from_numpy(p.A).to(dev) for p in probs]
    Bs = [torch.from_numpy(p.B).to(dev) for p in probs]
    fs = [binding.Factors(m, n, reverse=args.order == "reverse") for _ in range(N)]
    handles = [f.handle for f in fs]
    shapes = [(m, n)] * N
    Zs = [torch.empty((m, n), dtype=torch.int32, device=dev) for _ in range(N)]
    Ys = [torch.empty((m, n), dtype=Xs[0].dtype, device=dev) for _ in range(N)]
    obj = torch.empty(N, dtype=torch.float64, device=dev)
    ws = torch.empty(binding.gptq2d_round_batched_workspace_size(handles), dtype=torch.uint8, device=dev)
    fws = torch.empty(binding.gptq2d_factor_batched_workspace_size(N), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    # the argument arrays are built once (a loop over the same tensors)
    factor_call = binding.gptq2d_factor_batched(handles, As, Bs, fws, stream, shapes=shapes, prepare=True)
    round_call = binding.gptq2d_round_batched(handles, Xs, Zs, Ys, obj, ws, stream, shapes=shapes,
                                              prepare=True)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        factor_call()
        if ev is not None:
            ev[1].record(stream)
        round_call()
        if ev is not None:
            ev[2].record(stream)

    log(f"warmup {args.warmup}")
    for _ in range(max(args.warmup, 1)):
        step()
    binding.gptq2d_factor_batched_check(handles, stream)
    binding.gptq2d_round_batched_check(ws, stream)
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        step(ev[k])
    end.record(stream)
    torch.cuda.synchronize()
    binding.gptq2d_round_batched_check(ws, stream)
    ms_step = start.elapsed_time(end) / args.steps
    t_fac = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    t_round = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps
    out = {
        "metric": "rounded entries/s (a batch of problems per step)",
        "value": N * m * n / (ms_step * 1e-3),
        "unit": "entries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"{N} x c{args.config}: {WORKLOADS[args.config]}", "m": m, "n": n,
                   "batch": N, "io_dtype": probs[0].dtype, "order": args.order},
        "roofline": None,
        "phases_ms": {"factor": t_fac, "round": t_round},
        "round_entries_per_s": N * m * n / (t_round * 1e-3),
        "objective_sum": float(obj.sum().cpu()),
    }
    print(json.dumps(out), flush=True)
    for f in fs:
        f.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--dtype", default=None)
    ap.add_argument("--cpu-sample", type=int, default=2048)
    ap.add_argument("--cpu-sample-cols", type=int, default=512,
                    help="columns of the sample block the oracle's sweep is timed on")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--array-baseline", type=int, default=0, metavar="S",
                    help="also time the paper's own array-framework realisation (Algorithm 4 in "
                         "PyTorch) on the GPU on the leading S x S block")
    ap.add_argument("--array-block", type=int, default=64, metavar="W",
                    help="block width of that realisation")
    ap.add_argument("--batch", type=int, default=1, metavar="N",
                    help="N problems of the config (the layers of one model, each with its own X "
                         "and bases) per step, factorised and rounded by the batched entry points")
    ap.add_argument("--order", choices=["forward", "reverse"], default="forward",
                    help="rounding order: from the first row and column on, or from the last")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="run a plain MIB-MiB device copy first (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the library has no multi-GPU path).", file=sys.stderr, flush=True)
        sys.exit(2)

    import torch

    from paper_2607_27042_amd import binding, workloads as wl

    binding.load()  # raises when the HIP library is not built
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.batch > 1:
        run_batch(args, dev)
        return

    if args.copy_calibration > 0:
        log(f"copy calibration: {args.copy_calibration} MiB x 3")
        copy_calibration(args.copy_calibration)

    log(f"generating config {args.config}")
    prob = wl.make_config(args.config, args.dtype)
    m, n = prob.m, prob.n
    X = torch.from_numpy(prob.X).to(dev)
    A = torch.from_numpy(prob.A).to(dev)
    B = torch.from_numpy(prob.B).to(dev)
    f = binding.Factors(m, n, reverse=args.order == "reverse")
    ws = f.workspace()
    Z = torch.empty((m, n), dtype=torch.int32, device=dev)
    Y = torch.empty((m, n), dtype=X.dtype, device=dev)
    obj = torch.empty(1, dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        binding.gptq2d_factor_compute(f.handle, A, B, stream)
        binding.gptq2d_round(f.handle, X, Z, Y, obj, ws, stream)

    log(f"warmup {args.warmup}")
    for _ in range(max(args.warmup, 1)):
        step()
    binding.gptq2d_factor_check(f.handle, stream)
    binding.gptq2d_round_check(f.handle, ws, stream)
    torch.cuda.synchronize()

    def timed(instrument: bool):
        """K steps bracketed by a device synchronize on both sides; with
        instrument, every stage-kernel dispatch is also timed by HIP events
        that take the dispatch's own start / end stamps on the round's stream
        (this costs a few microseconds per dispatch, so the headline steps run
        without it)."""
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        binding.gptq2d_stage_timing(f.handle, instrument)
        start.record(stream)
        for k in range(args.steps):
            ev[k][0].record(stream)
            binding.gptq2d_factor_compute(f.handle, A, B, stream)
            ev[k][1].record(stream)
            binding.gptq2d_round(f.handle, X, Z, Y, obj, ws, stream)
            ev[k][2].record(stream)
        end.record(stream)
        torch.cuda.synchronize()
        res = {
            "ms_step": start.elapsed_time(end) / args.steps,
            "t_fac": sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps,
            "t_round": sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps,
        }
        binding.gptq2d_round_check(f.handle, ws, stream)
        res["stage_total_ms"], res["stage_launches"] = binding.gptq2d_stage_time(f.handle)
        binding.gptq2d_stage_timing(f.handle, False)
        return res

    log(f"timing {args.steps} steps")
    main_run = timed(False)
    log(f"timing {args.steps} steps with per-dispatch stage events")
    inst_run = timed(True)
    ms_step, t_fac, t_round = main_run["ms_step"], main_run["t_fac"], main_run["t_round"]
    stage_total_ms, stage_launches = inst_run["stage_total_ms"], inst_run["stage_launches"]

    stages = (m + 63) // 64 + (n + 63) // 64 - 1
    sweep_flop = m * n * (m + n)                      # m+n flop per rounded entry
    factor_flop_dense = (5.0 / 3.0) * (m ** 3 + n ** 3)
    # the Gram as formed on the envelope of these bases: the Cholesky and the
    # triangular inverse (d^3 / 3 each) plus the Gram's required products
    g0 = gram_flop(prob.A, 0, args.order == "reverse")
    g1 = gram_flop(prob.B, 1, args.order == "reverse")
    factor_flop = (2.0 / 3.0) * (m ** 3 + n ** 3) + g0[1] + g1[1]
    per_launch = sweep_flop / stages
    assert stage_launches == stages * args.steps, (stage_launches, stages, args.steps)
    stage_ms = stage_total_ms / stage_launches        # average stage-kernel launch (HIP events)
    achieved = per_launch / (stage_ms * 1e-3) / 1e12
    fac_tf = factor_flop / (t_fac * 1e-3) / 1e12
    value = m * n / (ms_step * 1e-3)

    out = {
        "metric": METRIC if args.config == 3 else f"rounded entries/s at the c{args.config} workload",
        "value": value,
        "unit": "entries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"c{args.config}: {WORKLOADS[args.config]}", "m": m, "n": n,
                   "io_dtype": prob.dtype, "order": args.order},
        "roofline": {
            "bound": "mfma", "achieved": achieved, "peak": PEAK_F64_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_F64_TFLOPS, "traffic": (stage_traffic(args.config, prob.dtype)
                                                          if args.order == "forward" else None),
            "frac_of_fp32_peak_reference": achieved / PEAK_F32_TFLOPS,
            "kernel": "k_stage (sweep stage: in-tile rounding + deferred-feedback GEMM tasks)",
            "flop_per_launch": per_launch, "launches_per_step": stages,
            "avg_launch_ms": stage_ms,
            "launch_timing": (f"HIP events on the dispatches of {stage_launches} stage launches "
                              f"({args.steps} further steps, round {inst_run['t_round']:.3f} ms "
                              f"with the events)"),
        },
        "phases_ms": {"factor": t_fac, "round": t_round},
        "round_entries_per_s": m * n / (t_round * 1e-3),
        "roofline_factor": {"bound": "mfma", "achieved": fac_tf, "peak": PEAK_F64_TFLOPS,
                            "unit": "TFLOP/s", "frac": fac_tf / PEAK_F64_TFLOPS,
                            "flop": factor_flop, "flop_dense": factor_flop_dense,
                            "flop_note": "Gram on the envelope of the bases (exact zeros skipped): "
                                         f"{(g0[1] + g1[1]) / (g0[0] + g1[0]):.3f} of the dense Gram"},
        "objective": float(obj.cpu()[0]),
    }
    if args.array_baseline > 0:
        log(f"array-framework realisation on the leading {args.array_baseline} block")
        out["array_baseline"] = array_baseline_run(prob, args.array_baseline, args.array_block, dev)
    if not args.no_cpu_baseline:
        log(f"cpu baseline on a {args.cpu_sample} sample")
        out["cpu_baseline"] = cpu_baseline(prob, args.cpu_sample, args.order == "reverse",
                                           args.cpu_sample_cols)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
