"""Benchmark of the element-wise merge/update hot path on one MI355X.

One step = the whole path over the 7B-shaped stack (28 layers of q/k/v/o/gate/up/down,
embedding and lm_head: 198 bf16 tensors, 7,615,283,200 parameters), K = 4 deltas, in one
call: TopKMask selection of every delta, sign election, disjoint mean and
theta_0 + lambda*tau (iso_update FUSED, TIES, lambda = 1, selection inside the call).  The
default single-read path reads each delta and the base once; --path two-pass times the
histogram select (iso_topk_mask) followed by the merge pass instead.  Inputs are synthetic
(seeded generator, written straight into HBM) and resident before timing.

Prints one JSON line.  Only one GPU is used; --gpus above 1 exits with a message.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
METRICS = {"7b": "merged params/sec and achieved HBM GB/s (% of peak), 7B-shaped K=4 merge",
           "1.5b": "merged params/sec and achieved HBM GB/s (% of peak), 1.5B-shaped K=4 merge",
           "layer": "merged params/sec and achieved HBM GB/s (% of peak), single bf16 layer K=2 merge",
           "7b-tsv": "merged params/sec and achieved HBM GB/s (% of peak), 7B-shaped K=4 merge with TSV on the "
                     "MLP matrices"}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = {"single-read": ("iso_fused.hip", "iso_merge_math.h", "iso_device.h"),
                  "two-pass": ("iso_merge.hip", "iso_merge_math.h", "iso_device.h")}
KERNEL_NAMES = {"single-read": "k_fs_main (single read: bracketed TopKMask + elect + disjoint mean + update)",
                "two-pass": "k_merge (elect + disjoint mean + update, thresholds known)"}


def kernel_source_hash(path):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[path]:
        h.update(open(os.path.join(ROOT, "paper_2607_19331_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(key, path):
    """HBM bytes per launch of the main kernel from the committed rocprofv3 counter runs,
    if they were taken on the current kernel source (else None)."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    r = rec.get(key)
    if not r or r.get("kernel_hash") != kernel_source_hash(path):
        return None
    return r.get("bytes_per_launch")


def _oracle_on_tensor(name, t, barrier=None):
    """One tensor of a workload through the oracle's TIES path (full-sort TopKMask, exact election,
    disjoint mean, update); returns (params, seconds of the oracle call, generation excluded).
    With a barrier, the call starts once every worker has its inputs."""
    import synth
    from oracle import ties
    wl = synth.workload(name)
    spec = wl.tensors[t]
    base = synth.fill_host(wl, t, 0)
    ds = [synth.fill_host(wl, t, 1 + i) for i in range(wl.K)]
    k = (spec.numel * wl.density.numerator * 2 + wl.density.denominator) // (2 * wl.density.denominator)
    if barrier is not None:
        barrier.wait()
    t0 = time.perf_counter()
    ties.merge_unit(base, ds, "bf16", "ties", k=k)
    return spec.numel, time.perf_counter() - t0


def _baseline_worker(name, t, barrier, queue):
    queue.put(_oracle_on_tensor(name, t, barrier))


# Bounded oracle samples per workload: (one-thread picks, all-cores picks), tensor indices.  The
# all-cores sample gives each worker one tensor, in table order.
BASELINE_PICKS = {
    "7b": ([1, 2, 0, 3, 4], list(range(16))),
    "1.5b": (list(range(7)), list(range(16))),
    "layer": ([0, 1], list(range(7))),
}


def cpu_baseline(name, workers):
    """The oracle, as it is, on a bounded sample of the same workload, on the host's cores: one
    thread over a few tensors; then `workers` processes (spawned, so that none inherits a GPU
    context) with one tensor each, started together once all have generated their inputs, the
    rate being their summed params over the slowest one's oracle time.  Runs before the
    benchmark touches the GPU."""
    import multiprocessing as mp
    import synth
    wl = synth.workload(name)
    one, many = BASELINE_PICKS[name]
    n1, dt1 = 0, 0.0
    for t in one:
        n, dt = _oracle_on_tensor(name, t)
        n1 += n
        dt1 += dt
    names1 = "+".join(sorted({wl.tensors[t].name.split(".")[-1] for t in one}))
    single = {"value": n1 / dt1, "unit": "params/s", "cores": 1, "kind": "oracle",
              "sample": f"{len(one)} tensors of layer 0 ({names1}; {n1} params, K={wl.K}) in {dt1:.1f} s; "
                        f"numpy, one thread"}
    picks = many[:workers]
    if len(picks) <= 1:
        return single, None
    ctx = mp.get_context("spawn")
    barrier, queue = ctx.Barrier(len(picks)), ctx.Queue()
    procs = [ctx.Process(target=_baseline_worker, args=(name, t, barrier, queue)) for t in picks]
    for p in procs:
        p.start()
    res = [queue.get() for _ in procs]
    for p in procs:
        p.join()
    nm_ = sum(r[0] for r in res)
    slowest = max(r[1] for r in res)
    allc = {"value": nm_ / slowest, "unit": "params/s", "cores": len(picks), "kind": "oracle",
            "sample": f"{len(picks)} tensors ({wl.tensors[picks[0]].name} .. {wl.tensors[picks[-1]].name}; {nm_} "
                      f"params, K={wl.K}), one per process, started together: summed params over the slowest "
                      f"oracle call ({slowest:.1f} s)"}
    return allc, single


def svd_flops(m, n):
    """Golub & Van Loan's operation count for the thin SVD with both factors (m >= n; U is m x n,
    as Algorithm 1 uses it): the cheaper of Golub-Reinsch, 14 m n^2 + 8 n^3, and R-SVD,
    6 m n^2 + 20 n^3."""
    m, n = max(m, n), min(m, n)
    return min(14 * m * n * n + 8 * n ** 3, 6 * m * n * n + 20 * n ** 3)


def bench_tiny(args, iso, synth, torch):
    """Tiny (fp32 256x256, K = 3): per step, the TIES update (selection inside the call) and
    ISO-Merger (Algorithm 1, iso_update SPECTRAL) on the same inputs, each timed with HIP
    events on the current stream.  The roofline is that of the SPECTRAL call: binary64, its
    algorithmic flops those of the K + 1 thin SVDs and the two polar SVDs it performs."""
    from oracle import numerics as nm
    from oracle import spectral as sp
    wl = synth.workload("tiny")
    spec = wl.tensors[0]
    n, K = spec.numel, wl.K
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    base = torch.empty(n, dtype=torch.int32, device=dev)
    synth.fill_device(base.data_ptr(), n, wl, 0, 0, stream)
    ds = []
    for i in range(K):
        d = torch.empty(n, dtype=torch.int32, device=dev)
        synth.fill_device(d.data_ptr(), n, wl, 0, 1 + i, stream)
        ds.append(d)
    out_t = torch.empty(n, dtype=torch.int32, device=dev)
    out_s = torch.empty(n, dtype=torch.int32, device=dev)
    k = iso.iso_k_from_density(n, wl.density.numerator, wl.density.denominator)
    et = [iso.Entry(spec.rows, spec.cols, base=base, deltas=ds, out=out_t, k=k)]
    es = [iso.Entry(spec.rows, spec.cols, base=base, deltas=ds, out=out_s, k=k)]
    ws_t = iso.workspace(iso.OP_UPDATE_FUSED_SELECT, et, K, iso.F32, dev)
    ws_s = iso.workspace(iso.OP_UPDATE_SPECTRAL, es, K, iso.F32, dev)

    def step(ev=None):
        if ev:
            ev[0].record()
        iso.iso_update(et, K, iso.F32, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, lam=1.0, desc=None, ws=ws_t)
        if ev:
            ev[1].record()
        iso.iso_update(es, K, iso.F32, iso.UPDATE_SPECTRAL, ws=ws_s)
        if ev:
            ev[2].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for w in (ws_t, ws_s):
        if iso.iso_read_device_status(w) != 0:
            raise RuntimeError("device status reports an error")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s_ in range(args.steps):
        step(ev[s_])
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    ties_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    spec_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps
    m_, n_ = spec.rows, spec.cols
    q = min(m_, n_)
    flops = (K + 1) * svd_flops(m_, n_) + svd_flops(m_, q) + svd_flops(n_, q)
    rec = {
        "metric": "ISO-Merger params/sec and FP64 TFLOP/s (% of peak), Tiny fp32 256x256 K=3",
        "value": n / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"Tiny: one fp32 {m_}x{n_} base, K={K} deltas (nonzero prob 0.3), TIES density "
                               f"{float(wl.density)}: TIES update and ISO-Merger (Algorithm 1) per step"},
        "ties_ms": ties_ms,
        "spectral_ms": spec_ms,
        "roofline": {"bound": "fp64", "kernel": "iso_update SPECTRAL (Algorithm 1: Jacobi SVDs, dense binary64 steps)",
                     "achieved": flops / (spec_ms * 1e-3) / 1e12, "peak": 78.6, "unit": "TFLOP/s",
                     "frac": flops / (spec_ms * 1e-3) / 1e12 / 78.6, "traffic": None,
                     "flops_per_call": flops},
    }
    if not args.no_cpu_baseline:
        w0 = nm.to_f64(synth.fill_host(wl, 0, 0), "f32").reshape(m_, n_)
        dh = [nm.to_f64(synth.fill_host(wl, 0, 1 + i), "f32").reshape(m_, n_) for i in range(K)]
        reps, t1 = 0, time.perf_counter()
        while reps < 3 or time.perf_counter() - t1 < 10.0:
            sp.iso_merge(w0, dh)
            reps += 1
        dt = (time.perf_counter() - t1) / reps
        try:
            from threadpoolctl import threadpool_info
            cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        except ImportError:
            cores = len(os.sched_getaffinity(0))
        rec["cpu_baseline"] = {"value": n / dt, "unit": "params/s", "cores": cores,
                               "kind": "oracle",
                               "sample": f"Algorithm 1 (LAPACK SVDs, numpy) on the whole Tiny matrix, {reps} runs, "
                                         f"{dt * 1e3:.1f} ms each"}
    return rec


SPECTRAL_SETS = {
    # config: (workload, tensor indices, description)
    "layer-spectral": ("layer", list(range(7)), "single bf16 layer (q/k/v/o 2048x2048, gate/up 2048x5632, "
                                                 "down 5632x2048)"),
    "7b-layer-spectral": ("7b", list(range(7)), "one full 7B layer (q/o 3584x3584, k/v 512x3584, gate/up "
                                                 "18944x3584, down 3584x18944)"),
    "7b-embed-spectral": ("7b", [196], "the 7B embedding matrix (152064x3584)"),
}


def bench_layer_spectral(args, iso, synth, torch):
    """ISO-Merger (Algorithm 1, iso_update SPECTRAL) over a set of bf16 matrices with the workload's
    K deltas in one call per step, timed with HIP events on the current stream: the single layer
    (K = 2), one full layer of the 7B stack or its embedding matrix (K = 4).  Roofline: binary64, the
    algorithmic flops of every matrix's K + 1 thin SVDs and two polar SVDs."""
    from oracle import numerics as nm
    from oracle import spectral as sp
    wl_name, picks, what = SPECTRAL_SETS[args.config]
    wl = synth.workload(wl_name)
    K = wl.K
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    entries, flops, N = [], 0, 0
    for t in picks:
        spec = wl.tensors[t]
        n = spec.numel
        N += n
        base = torch.empty(n, dtype=torch.int16, device=dev)
        synth.fill_device(base.data_ptr(), n, wl, t, 0, stream)
        ds = []
        for i in range(K):
            d = torch.empty(n, dtype=torch.int16, device=dev)
            synth.fill_device(d.data_ptr(), n, wl, t, 1 + i, stream)
            ds.append(d)
        out = torch.empty(n, dtype=torch.int16, device=dev)
        entries.append(iso.Entry(spec.rows, spec.cols, base=base, deltas=ds, out=out, k=0))
        m_, n_ = spec.rows, spec.cols
        q = min(m_, n_)
        flops += (K + 1) * svd_flops(m_, n_) + svd_flops(m_, q) + svd_flops(n_, q)
    ws = iso.workspace(iso.OP_UPDATE_SPECTRAL, entries, K, iso.BF16, dev)

    def step():
        iso.iso_update(entries, K, iso.BF16, iso.UPDATE_SPECTRAL, ws=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if iso.iso_read_device_status(ws) != 0:
        raise RuntimeError("device status reports an error")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s_ in range(args.steps):
        ev[s_][0].record()
        step()
        ev[s_][1].record()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    spec_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    rec = {
        "metric": f"ISO-Merger params/sec and FP64 TFLOP/s (% of peak), {what.split(' (')[0]} K={K}",
        "value": N / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{what}: {len(picks)} matrices, {N} params, K={K} deltas "
                               f"({float(wl.delta.p_zero):.0%} zeros): ISO-Merger (Algorithm 1) in one call"},
        "spectral_ms": spec_ms,
        "roofline": {"bound": "fp64", "kernel": "iso_update SPECTRAL (Algorithm 1: Jacobi SVDs, dense binary64 steps)",
                     "achieved": flops / (spec_ms * 1e-3) / 1e12, "peak": 78.6, "unit": "TFLOP/s",
                     "frac": flops / (spec_ms * 1e-3) / 1e12 / 78.6, "traffic": None,
                     "flops_per_call": flops},
    }
    if not args.no_cpu_baseline:
        t = min(picks, key=lambda j: wl.tensors[j].numel)        # the smallest matrix of the set
        spec = wl.tensors[t]
        rows = min(spec.rows, 8192)                                # a 152064-row matrix: its first rows
        n = rows * spec.cols
        w0 = nm.to_f64(synth.fill_host(wl, t, 0, n=n), "bf16").reshape(rows, spec.cols)
        dh = [nm.to_f64(synth.fill_host(wl, t, 1 + i, n=n), "bf16").reshape(rows, spec.cols) for i in range(K)]
        t1 = time.perf_counter()
        sp.iso_merge(w0, dh)
        dt = time.perf_counter() - t1
        try:
            from threadpoolctl import threadpool_info
            cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        except ImportError:
            cores = len(os.sched_getaffinity(0))
        part = "" if rows == spec.rows else f", its first {rows} rows as one matrix"
        rec["cpu_baseline"] = {"value": n / dt, "unit": "params/s", "cores": cores, "kind": "oracle",
                               "sample": f"Algorithm 1 (LAPACK SVDs, numpy) on {spec.name} "
                                         f"({spec.rows}x{spec.cols}{part}), one run, {dt:.1f} s"}
    return rec


ORTHO_SETS = {
    # config: (workload, tensor indices, description); OrthoMerge needs rows >= cols
    "layer-ortho": ("layer", [0, 1, 2, 3, 6], "single bf16 layer, its tall and square matrices (q/k/v/o "
                                               "2048x2048, down 5632x2048)"),
    "7b-layer-ortho": ("7b", [0, 3, 4, 5], "one 7B layer, its tall and square matrices (q/o 3584x3584, "
                                            "gate/up 18944x3584)"),
}


def ortho_flops(m, n, K):
    """Work OrthoMerge-G-TIES prescribes per matrix: Golub & Van Loan's SVD count for each of the K
    Procrustes SVDs of W_0^T W_i, 2 m n^2 for each product with W_0 (W_0^T W_i, W_0 R_i, W_0 R),
    and 8/3 n^3 for each of the K + 1 Cayley solves with n right-hand sides (LU, then two
    triangular solves)."""
    return K * svd_flops(n, n) + (2 * K + 1) * 2 * m * n * n + (K + 1) * 8 * n ** 3 // 3


def bench_ortho(args, iso, synth, torch):
    """OrthoMerge-G-TIES (App. F; iso_update ORTHO) over a set of bf16 matrices with the workload's
    K deltas in one call per step, residual TopKMask density 0.2 (the paper's setting), lambda 1;
    timed with HIP events.  Roofline: binary64, the algorithmic flops of ortho_flops."""
    from oracle import numerics as nm
    from oracle import orthomerge as om
    wl_name, picks, what = ORTHO_SETS[args.config]
    wl = synth.workload(wl_name)
    K = wl.K
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    entries, flops, N = [], 0, 0
    for t in picks:
        spec = wl.tensors[t]
        n = spec.numel
        N += n
        base = torch.empty(n, dtype=torch.int16, device=dev)
        synth.fill_device(base.data_ptr(), n, wl, t, 0, stream)
        ds = []
        for i in range(K):
            d = torch.empty(n, dtype=torch.int16, device=dev)
            synth.fill_device(d.data_ptr(), n, wl, t, 1 + i, stream)
            ds.append(d)
        out = torch.empty(n, dtype=torch.int16, device=dev)
        k = iso.iso_k_from_density(n, 1, 5)
        entries.append(iso.Entry(spec.rows, spec.cols, base=base, deltas=ds, out=out, k=k))
        flops += ortho_flops(spec.rows, spec.cols, K)
    ws = iso.workspace(iso.OP_UPDATE_ORTHO, entries, K, iso.BF16, dev)

    def step():
        iso.iso_update(entries, K, iso.BF16, iso.UPDATE_ORTHO, lam=1.0, ws=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if iso.iso_read_device_status(ws) != 0:
        raise RuntimeError("device status reports an error")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s_ in range(args.steps):
        ev[s_][0].record()
        step()
        ev[s_][1].record()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    call_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    rec = {
        "metric": f"OrthoMerge-G-TIES params/sec and FP64 TFLOP/s (% of peak), {what.split(',')[0]} K={K}",
        "value": N / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{what}: {len(picks)} matrices, {N} params, K={K} deltas "
                               f"({float(wl.delta.p_zero):.0%} zeros), residual TopKMask density 0.2, lambda 1: "
                               f"OrthoMerge-G-TIES in one call"},
        "call_ms": call_ms,
        "roofline": {"bound": "fp64", "kernel": "iso_update ORTHO (Jacobi SVDs, dense binary64 steps, TIES)",
                     "achieved": flops / (call_ms * 1e-3) / 1e12, "peak": 78.6, "unit": "TFLOP/s",
                     "frac": flops / (call_ms * 1e-3) / 1e12 / 78.6, "traffic": None, "flops_per_call": flops},
    }
    if not args.no_cpu_baseline:
        t = picks[0]
        spec = wl.tensors[t]
        rows, cols = min(spec.rows, 2048), min(spec.cols, 2048)
        w0 = synth.fill_host(wl, t, 0).reshape(spec.rows, spec.cols)[:rows, :cols]
        dh = [synth.fill_host(wl, t, 1 + i).reshape(spec.rows, spec.cols)[:rows, :cols] for i in range(K)]
        t1 = time.perf_counter()
        om.orthomerge_ties(w0, dh, nm.k_from_density(rows * cols, 0.2), dtype="bf16")
        dt = time.perf_counter() - t1
        try:
            from threadpoolctl import threadpool_info
            cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        except ImportError:
            cores = len(os.sched_getaffinity(0))
        part = "" if (rows, cols) == (spec.rows, spec.cols) else f", its leading {rows}x{cols} block as one matrix"
        rec["cpu_baseline"] = {"value": rows * cols / dt, "unit": "params/s", "cores": cores, "kind": "oracle",
                               "sample": f"OrthoMerge-G-TIES (LAPACK SVD, numpy) on {spec.name} "
                                         f"({spec.rows}x{spec.cols}{part}), one run, {dt:.1f} s"}
    return rec


def bench_layer_optimizer(args, iso, synth, torch):
    """One ISO-AdamW step (iso_optimizer_step) or, with --rule muon, one ISO-Muon step
    (iso_optimizer_step_muon) over the single layer's seven matrices (q/k/v/o 2048x2048, gate/up
    2048x5632, down 5632x2048) with full-rank frames, bf16 weights and gradients, timed with HIP
    events.  Roofline: the dominant work, the Newton-Schulz polar iterations (binary64 MFMA
    products): the flops their steps performed, as the library counts them, over their time
    from the library's profiling events in the same run."""
    import numpy as np
    from oracle import optimizer as op
    wl = synth.workload("layer")
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    frames = []
    for t, spec in enumerate(wl.tensors):
        m, n = spec.rows, spec.cols
        q = min(m, n)
        u, _ = torch.linalg.qr(torch.randn(m, q, dtype=torch.float64, device=dev, generator=gen))
        v, _ = torch.linalg.qr(torch.randn(n, q, dtype=torch.float64, device=dev, generator=gen))
        s = torch.sort(torch.rand(q, dtype=torch.float64, device=dev, generator=gen) + 0.5, descending=True)[0]
        grad = torch.empty(m * n, dtype=torch.int16, device=dev)
        synth.fill_device(grad.data_ptr(), m * n, wl, t, 1, stream)     # delta-shaped values as G_W
        z = lambda r: torch.zeros(r * q, dtype=torch.float64, device=dev)
        frames.append(iso.Frame(u=u.t().contiguous().view(-1), v=v.t().contiguous().view(-1), sigma=s,
                                m_u=z(m), v_u=z(m), m_v=z(n), v_v=z(n), grad=grad,
                                w_out=torch.empty(m * n, dtype=torch.int16, device=dev), rows=m, cols=n, rank=q))
    ws = iso.optimizer_workspace(frames, dev)
    muon = args.rule == "muon"
    hp = dict(lr=1e-6, weight_decay=0.0) if muon else dict(lr=1e-6, beta1=0.9, beta2=0.999, eps=1e-8,
                                                          weight_decay=0.0)
    name = "ISO-Muon" if muon else "ISO-AdamW"
    step_no = [0]

    def step():
        step_no[0] += 1
        if muon:
            iso.iso_optimizer_step_muon(frames, iso.BF16, momentum=0.95, nesterov=True, ws=ws, **hp)
        else:
            iso.iso_optimizer_step(frames, iso.BF16, step=step_no[0], ws=ws, **hp)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if iso.iso_read_device_status(ws) != 0:
        raise RuntimeError("device status reports an error")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    iso.iso_profile_begin()
    t0 = time.perf_counter()
    for s_ in range(args.steps):
        ev[s_][0].record()
        step()
        ev[s_][1].record()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    ns_flops = iso.iso_profile_flops()
    ns_ms, ns_regions = iso.iso_profile_end()
    opt_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    N = wl.numel
    rec = {
        "metric": f"{name} step params/sec and FP64 TFLOP/s (% of peak), single bf16 layer",
        "value": N / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"single bf16 layer ({len(wl.tensors)} matrices, {N} params): one {name} step "
                               f"(factor gradients, {'Muon with polar directions' if muon else 'AdamW'}, polar "
                               "retraction, W+) on full-rank frames"},
        "optimizer_ms": opt_ms,
        "newton_schulz_ms": ns_ms / args.steps,
        "roofline": {"bound": "fp64", "kernel": "Newton-Schulz polar iterations (k_gemm_jobs binary64 MFMA "
                     "products with their step kernels; " + ("directions and retraction" if muon else "retraction") +
                     f", {ns_regions // args.steps} per step)",
                     "achieved": ns_flops / (ns_ms * 1e-3) / 1e12, "peak": 78.6, "unit": "TFLOP/s",
                     "frac": ns_flops / (ns_ms * 1e-3) / 1e12 / 78.6, "traffic": None,
                     "flops_per_call": ns_flops / args.steps},
    }
    if not args.no_cpu_baseline:
        spec = wl.tensors[0]
        m, n = spec.rows, spec.cols
        rng = np.random.default_rng(0)
        u0, _ = np.linalg.qr(rng.standard_normal((m, m)))
        v0, _ = np.linalg.qr(rng.standard_normal((n, n)))
        s0 = np.sort(rng.uniform(0.5, 1.5, m))[::-1]
        g = rng.standard_normal((m, n)) * 1e-4
        t1 = time.perf_counter()
        if muon:
            op.iso_muon_step(u0, v0, s0, g, (np.zeros((m, m)), np.zeros((n, m))), 1e-6, 0.95)
        else:
            op.iso_adamw_step(u0, v0, s0, g, tuple(np.zeros((r, m)) for r in (m, m, n, n)), 1, 1e-6)
        dt = time.perf_counter() - t1
        try:
            from threadpoolctl import threadpool_info
            cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        except ImportError:
            cores = len(os.sched_getaffinity(0))
        rec["cpu_baseline"] = {"value": spec.numel / dt, "unit": "params/s", "cores": cores, "kind": "oracle",
                               "sample": f"one {name} step (LAPACK polar, numpy) on {spec.name} ({m}x{n}), {dt:.1f} s"}
    return rec


def calibrate_stream(args, torch):
    """Rate of the fused pass's traffic mix with trivial arithmetic: libiso_calibrate's kernel reads
    K + 1 = 5 arrays of the 7B stack's size (7,615,283,200 bf16 each) and writes one, with the main
    pass's launch shape; then the 5 reads alone, then a 1:1 copy.  HIP events on the current stream."""
    import ctypes
    import synth
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2607_19331_amd", "libiso_calibrate.so"))
    lib.iso_calibrate_stream.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_int, ctypes.c_void_p]
    n = synth.stack_7b().numel
    n_vec = n // 8
    arrs = [torch.full((n_vec * 8,), i + 1, dtype=torch.int16, device="cuda:0") for i in range(6)]
    stream = torch.cuda.current_stream()
    res = {}
    for name, n_in, write in (("5_read_1_write", 5, 1), ("5_read", 5, 0), ("1_read_1_write", 1, 1)):
        ptrs = (ctypes.c_void_p * 8)(*[a.data_ptr() for a in arrs[:n_in]])
        out = arrs[5].data_ptr()
        for _ in range(2):
            if lib.iso_calibrate_stream(ptrs, n_in, out, n_vec, write, stream.cuda_stream) != 0:
                raise RuntimeError("iso_calibrate_stream failed")
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        reps = 5
        ev[0].record()
        for _ in range(reps):
            lib.iso_calibrate_stream(ptrs, n_in, out, n_vec, write, stream.cuda_stream)
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / reps
        nbytes = n_vec * 16 * (n_in + write)
        res[name] = {"ms": ms, "bytes": nbytes, "GBps": nbytes / (ms * 1e-3) / 1e9,
                     "frac_of_8TBps": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS}
    return {"calibrate_stream": res, "elements_per_array": n_vec * 8}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="7b", choices=["tiny", "layer", "1.5b", "7b", "7b-tsv", "layer-optimizer"]
                    + list(SPECTRAL_SETS) + list(ORTHO_SETS))
    ap.add_argument("--path", default="single-read", choices=["single-read", "two-pass"])
    ap.add_argument("--lam", type=float, default=1.0,
                    help="lambda of the stack configs' TIES update (the paper's TIES: 1; other values take the "
                         "general binary64 rounding path of the fused pass)")
    ap.add_argument("--select", default="per-tensor", choices=["per-tensor", "whole-model"],
                    help="whole-model: one TopKMask over the concatenation of every tensor's delta (all "
                         "tensors in one select_group; the two-pass path)")
    ap.add_argument("--rule", default="adamw", choices=["adamw", "muon"],
                    help="base rule of the ISO-Optimizer step (--config layer-optimizer)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain elementwise copy (1 GiB read, 1 GiB written, 3 launches) to scale "
                         "the HBM byte counters of a profiler")
    ap.add_argument("--calibrate-stream", action="store_true",
                    help="run only the streaming calibration kernel over the 7B stack's arrays (K deltas + base "
                         "read, weights written; then reads only; then a copy) and print the rates")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the merge path is independent per "
              "tensor and is not sharded across GPUs here.", file=sys.stderr)
        sys.exit(2)

    # the oracle baseline of the stack workloads runs first, in processes spawned before anything
    # in this one touches the GPU
    baseline = None
    # (the whole-model selection has no bounded oracle sample: its threshold needs every tensor)
    if not args.no_cpu_baseline and args.config in BASELINE_PICKS and args.select == "per-tensor" and not (
            args.calibrate_copy or args.calibrate_stream):
        workers = min(len(os.sched_getaffinity(0)), 16, len(BASELINE_PICKS[args.config][1]))
        baseline = cpu_baseline(args.config, workers)

    import torch

    if args.calibrate_copy:
        n = 1 << 29                                 # 2-byte elements: 1 GiB each way
        src = torch.ones(n, dtype=torch.float16, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy": {"bytes_read": 2 * n, "bytes_written": 2 * n, "launches": 3}}), flush=True)
        return

    if args.calibrate_stream:
        print(json.dumps(calibrate_stream(args, torch)), flush=True)
        return

    import paper_2607_19331_amd as iso
    import synth

    if args.config == "tiny":
        print(json.dumps(bench_tiny(args, iso, synth, torch)), flush=True)
        return
    if args.config in ORTHO_SETS:
        print(json.dumps(bench_ortho(args, iso, synth, torch)), flush=True)
        return
    if args.config in SPECTRAL_SETS:
        print(json.dumps(bench_layer_spectral(args, iso, synth, torch)), flush=True)
        return
    if args.config == "layer-optimizer":
        print(json.dumps(bench_layer_optimizer(args, iso, synth, torch)), flush=True)
        return

    wl = synth.workload(args.config)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    K = wl.K
    entries, tsv_entries = [], []
    for t, spec in enumerate(wl.tensors):
        n = spec.numel
        base = torch.empty(n, dtype=torch.int16, device=dev)
        synth.fill_device(base.data_ptr(), n, wl, t, 0, stream)
        ds = []
        for i in range(K):
            d = torch.empty(n, dtype=torch.int16, device=dev)
            synth.fill_device(d.data_ptr(), n, wl, t, 1 + i, stream)
            ds.append(d)
        out = torch.empty(n, dtype=torch.int16, device=dev)
        k = iso.iso_k_from_density(n, wl.density.numerator, wl.density.denominator)
        e = iso.Entry(spec.rows, spec.cols, base=base, deltas=ds, out=out, k=k)
        if wl.tsv_rank and spec.name.split(".")[-1] in wl.tsv_names:
            tsv_entries.append(e)
        else:
            entries.append(e)
    N = wl.numel
    whole = args.select == "whole-model"
    if whole:
        for e in entries:
            e.group = 1
        args.path = "two-pass"
    single = args.path == "single-read"
    if single:
        ws_upd = iso.workspace(iso.OP_UPDATE_FUSED_SELECT, entries, K, iso.BF16, dev)
        ws_sel, desc = None, None
    else:
        desc = iso.desc_tensor(len(entries) * K, dev)
        ws_sel = iso.workspace(iso.OP_TOPK, entries, K, iso.BF16, dev)
        ws_upd = iso.workspace(iso.OP_UPDATE_FUSED, entries, K, iso.BF16, dev)
    ws_tsv = iso.workspace(iso.OP_BLOCKDIAG, tsv_entries, K, iso.BF16, dev, rank=wl.tsv_rank) if tsv_entries else None
    torch.cuda.synchronize()

    def step(ev=None):
        if ev:
            ev[0].record()
        if not single:
            iso.iso_topk_mask(entries, K, iso.BF16, desc, ws=ws_sel)
        iso.iso_update(entries, K, iso.BF16, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, lam=args.lam, desc=desc,
                       ws=ws_upd)
        if ev:
            ev[1].record()
        if tsv_entries:
            iso.iso_blockdiag_project(tsv_entries, K, iso.BF16, wl.tsv_rank, 1.0, ws=ws_tsv)
        if ev:
            ev[2].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for w in (ws_sel, ws_upd, ws_tsv):
        if w is not None and iso.iso_read_device_status(w) != 0:
            raise RuntimeError("device status reports an error")
    fallbacks = iso.iso_read_fallback_count(ws_upd) if single else None
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    iso.iso_profile_begin()                     # HIP events around the main kernel, on this stream
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(ev[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    main_total, launches = iso.iso_profile_end()
    if launches != args.steps:
        raise RuntimeError(f"timed {launches} main-kernel launches for {args.steps} steps")
    main_ms = main_total / launches
    merge_call_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    tsv_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps
    ms_per_step = wall * 1e3 / args.steps

    n_elem = sum(e.rows * e.cols for e in entries)
    alg_bytes_step = N * (K * 2 + 2 + 2)            # each delta and the base read once, weights written once
    main_alg = n_elem * (K * 2 + 2 + 2)             # the main kernel's algorithmic bytes per launch
    main_gbps = main_alg / (main_ms * 1e-3) / 1e9
    what = "TopKMask select + elect + disjoint mean + update in one call"
    if whole:
        what = ("TopKMask over the whole-model delta (all tensors in one select_group), then elect + disjoint mean "
                "+ update")
    if tsv_entries:
        what += f"; TSV rank {wl.tsv_rank} on the {len(tsv_entries)} MLP matrices"
    rec = {
        "metric": METRICS[args.config] + (", whole-model TopKMask" if whole else "")
        + ("" if args.lam == 1.0 else f", lambda {args.lam:g}"),
        "value": N / (ms_per_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}-shaped stack: {len(wl.tensors)} bf16 tensors, {N} params, K={K} deltas "
                               f"({float(wl.delta.p_zero):.0%} zeros), TIES density {float(wl.density)} "
                               f"{'of the whole model' if whole else 'per tensor'}, lambda {args.lam:g}: {what}",
                   "path": args.path},
        "algorithmic_gbps": alg_bytes_step / (ms_per_step * 1e-3) / 1e9,
        "hbm_frac_step": alg_bytes_step / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBPS,
        "merge_call_ms": merge_call_ms,
        "main_kernel_ms": main_ms,
        "roofline": {"bound": "hbm", "kernel": KERNEL_NAMES[args.path],
                     "achieved": main_gbps, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": main_gbps / PEAK_HBM_GBPS,
                     "traffic": None if whole else measured_traffic(f"{args.config}/{args.path}", args.path)},
    }
    if single:
        rec["fallback_tensors"] = fallbacks
    if tsv_entries:
        rec["tsv_ms"] = tsv_ms
    if baseline is not None:
        rec["cpu_baseline"] = baseline[0]
        if baseline[1] is not None:
            rec["cpu_baseline_one_thread"] = baseline[1]
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
