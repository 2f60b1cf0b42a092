#!/usr/bin/env python3
"""Throughput of online SOM training on one MI355X.

One bench step is one pass of the whole hot path over the workload:
reset the map to its seeded initial prototypes, train it for the workload's
full schedule (epochs * n per-sample steps in one persistent kernel), then
assign every sample to its BMU and compute QE and TE (one batched MFMA BMU
search, som_evaluate).  Data, order and initial prototypes are resident in
HBM before timing starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload I] [--input csr]

prints one JSON line.  The default workload is the largest one, the
100,000 x 2048 Gaussian mixture on a 100 x 100 map; the line also carries
the 20,000 x 10,000 TF-IDF workload on a 50 x 50 map (`also`), the other
workload the memory target is set on, timed over a few passes.  `value` is
prototype*dim updates per second of the whole step, T * N * d / step time.

`roofline` reports the training call: algorithmic bytes 3 * N * d * 4 per
sample (read the prototypes for the distance, read and write them for the
update) divided by the average duration of som_train's kernels from HIP
events on their stream, against the 8 TB/s HBM peak (`frac`).  The blocked
kernels move fewer bytes than that model (W streams once per block of
steps, some rows stay in LDS), so `frac` can exceed 1; the memory the
kernel really moves is `traffic` (FETCH_SIZE + WRITE_SIZE counters of the
same kernel source, stored under profiles/), and `frac_applicable` is that
traffic's rate against `stream_inplace`, an in-place stream over a buffer
of W's size on the training grid measured in the same run.  `bound` comes
from the launch plan: the LDS-resident kernels never stream W and wait on
the grid exchange ("latency"), the streamed ones stream W once per block
("hbm").
`cpu_baseline` times the fp64 oracle on the host over a bounded prefix of
the same training run.
"""
import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "train_kernel_traffic.json")
TRAIN_SOURCES = [os.path.join(ROOT, "paper_1905_09598_amd", "csrc", f)
                 for f in ("som_device.h", "som_internal.h", "som_train.hip",
                           "som_train_pipe.h", "som_train_pipe.hip",
                           "som_train_pipe_stream.hip")]


def kernel_source_sha() -> str:
    """sha256 over the training kernels' sources (in a fixed order)."""
    h = hashlib.sha256()
    for path in TRAIN_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """Counter-measured HBM bytes per launch, if taken on this kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    ent = rec.get(workload)
    if not ent or ent.get("kernel_sha256") != kernel_source_sha():
        return None
    return ent.get("bytes_per_launch")


def cpu_baseline(cfg, X, order, budget_s: float, threads: int = 0):
    """fp64 oracle on the host over a prefix of the same training run, on
    `threads` OpenMP threads (0: every core this process may use)."""
    import numpy as np
    import oracle

    threads = threads or oracle.default_threads()
    W = oracle.init_uniform(cfg.init_seed, cfg.units, cfg.d)
    s = oracle.schedule(cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                        oracle.LINEAR, oracle.EXPONENTIAL)
    done, chunk = 0, 200
    t0 = time.perf_counter()
    while done < cfg.steps and time.perf_counter() - t0 < budget_s:
        k = min(chunk, cfg.steps - done)
        W, _ = oracle.train(W, cfg.rows, cfg.cols, X, order[done:done + k], s,
                            step0=done, total_steps=cfg.steps, nthreads=threads)
        done += k
    dt = time.perf_counter() - t0
    del np
    return {
        "value": done * cfg.units * cfg.d / dt,
        "unit": "proto*dim updates/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"first {done} of {cfg.steps} training steps of {cfg.name} "
                  f"(fp64, {threads} OpenMP threads, {dt:.1f} s)",
    }


def stream_inplace(nbytes: int, grid: int, target_ms: float = 40.0, reps: int = 3) -> dict:
    """In-place stream over one device buffer of nbytes (som_stream_inplace:
    each of `grid` workgroups reads and rewrites its own contiguous share,
    many passes in one launch, no gaps), best of reps, HIP events on the
    current stream.  A memory reference for the roofline, not a SOM step."""
    import torch

    import paper_1905_09598_amd as som

    nbytes = max(16, nbytes // 16 * 16)
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    st = torch.cuda.current_stream()
    som.som_stream_inplace(buf, nbytes, 1, grid, st.cuda_stream)
    # one pass moves 2 * nbytes; size the launch to about target_ms at 6 TB/s
    passes = max(1, int(target_ms * 1e-3 * 6e12 / (2 * nbytes)))
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        som.som_stream_inplace(buf, nbytes, passes, grid, st.cuda_stream)
        e1.record(st)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    moved = 2.0 * nbytes * passes
    del buf
    return {"bytes": nbytes, "passes": passes, "grid": grid, "ms": best,
            "GB/s": moved / (best / 1e3) / 1e9}


def host_cpu() -> dict:
    """The host's CPU model, physical cores and the cores this process may use."""
    model, cores = None, set()
    try:
        phys = core = None
        with open("/proc/cpuinfo") as f:
            for line in f:
                k, _, v = line.partition(":")
                k, v = k.strip(), v.strip()
                if k == "model name" and model is None:
                    model = v
                elif k == "physical id":
                    phys = v
                elif k == "core id":
                    core = v
                elif not k and phys is not None and core is not None:
                    cores.add((phys, core))
                    phys = core = None
    except OSError:
        pass
    try:
        allowed = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        allowed = os.cpu_count()
    return {"cpu_model": model, "physical_cores": len(cores) or None,
            "sockets": len({p for p, _ in cores}) or None, "allowed_cores": allowed}


def map_sweep(cpu_budget: float):
    """Per-step training time against map size at d = 64: an analogue of the
    paper's Table 3 (time against map size), on synthetic data: n = 8192
    samples of a 16-cluster Gaussian mixture (sd 0.2), one epoch, lr 0.5 ->
    0.01 linear, sigma side/2 -> 1 exponential, seeded as the workloads are."""
    import torch

    import oracle
    import paper_1905_09598_amd as som
    import workloads

    n, d = 8192, 64
    X = workloads.gaussian_mixture(n, d, 16, 0.2, seed=7)
    order = workloads.epoch_orders(n, 1, 7)
    Xd = torch.from_numpy(X).cuda()
    od = torch.from_numpy(order).cuda()
    stream = torch.cuda.current_stream()
    for side in (16, 32, 64, 128, 256, 512):
        N = side * side
        m = som.Map(side, side, d, seed=0)
        plan = m.plan()
        kw = dict(order=od)
        m.train(Xd, 1, 0.5, 0.01, side / 2.0, 1.0, **kw)  # warm-up
        times = []
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            m.train(Xd, 1, 0.5, 0.01, side / 2.0, 1.0, **kw)
            b.record(stream)
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b) / 1e3)
        t = sorted(times)[1]
        line = {"map": f"{side}x{side}", "units": N, "d": d, "steps": n,
                "us_per_step": t / n * 1e6, "proto_dim_updates_per_s": n * N * d / t,
                "train_s": t, "grid": plan["grid"],
                "variant": ["stream", "lds", "pipelined-stream", "pipelined-lds",
                            "pipelined-stream-cols"][plan["variant"]]}
        if cpu_budget > 0:
            W = oracle.init_uniform(0, N, d)
            s_ = oracle.schedule(0.5, 0.01, side / 2.0, 1.0)
            threads = oracle.default_threads()
            done, t0 = 0, time.perf_counter()
            while done < n and time.perf_counter() - t0 < cpu_budget / 6:
                k = min(100, n - done)
                W, _ = oracle.train(W, side, side, X, order[done:done + k], s_, step0=done,
                                    total_steps=n, nthreads=threads)
                done += k
            dt = time.perf_counter() - t0
            line["oracle_us_per_step"] = dt / done * 1e6
            line["oracle_cores"] = threads
        print(json.dumps(line), flush=True)
        m.close()


def batch_map_epoch(workload: int, steps: int, warmup: int):
    """Milliseconds per batch-map epoch (som_train_batch at the workload's
    starting radius), HIP events on the map's stream."""
    import torch

    import paper_1905_09598_amd as som
    import workloads

    cfg = workloads.WORKLOADS[workload]
    Xd = torch.from_numpy(workloads.make_data(cfg)).cuda()
    m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=cfg.init_seed)
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        m.train_batch(Xd, 1, cfg.sigma0, cfg.sigma0)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for a, b in ev:
        a.record(stream)
        m.train_batch(Xd, 1, cfg.sigma0, cfg.sigma0)
        b.record(stream)
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in ev)[len(ev) // 2]
    bmu_flops = 2.0 * cfg.n * cfg.units * cfg.d
    print(json.dumps({
        "metric": "batch-map epoch time (BMU of every sample, fp64 neighbourhood means)",
        "value": ms, "unit": "ms per epoch", "higher_is_better": False, "steps": steps,
        "data": "synthetic", "config": {"workload": cfg.name, "n": cfg.n, "d": cfg.d,
                                        "map": f"{cfg.rows}x{cfg.cols}", "sigma": cfg.sigma0},
        "bmu_flops_per_epoch": bmu_flops,
        "epoch_tflops_bmu_equivalent": bmu_flops / (ms / 1e3) / 1e12,
    }), flush=True)
    m.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=4,
                    help="index into the workload table (default: the 100,000 x 2048 "
                         "mixture on a 100 x 100 map)")
    ap.add_argument("--also", type=str, default="3",
                    help="comma-separated workload indices timed after the main one and "
                         "reported under `also` ('' for none)")
    ap.add_argument("--also-steps", type=int, default=3,
                    help="timed passes of each `also` workload (after one warm-up)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle time for the CPU baseline (0 = skip)")
    ap.add_argument("--map-sweep", action="store_true",
                    help="instead of the bench line: per-step time of training maps of "
                         "16x16 ... 512x512 units at d = 64 (one JSON line per map size)")
    ap.add_argument("--batch-map", action="store_true",
                    help="instead of the bench line: time one batch-map epoch "
                         "(som_train_batch) on the workload, one JSON line")
    ap.add_argument("--input", choices=("dense", "csr"), default="dense",
                    help="train from the dense rows (som_train) or from their CSR form "
                         "(som_train_csr, the sparse-input path)")
    ap.add_argument("--shard", type=int, default=1, metavar="G",
                    help="train one GPU's share of the workload's map when its prototype "
                         "rows are split over G GPUs: N / G units (as near-square a map as "
                         "divides N / G), the same samples, d and schedule; the arg-min "
                         "exchange between GPUs is not built, so this is the per-GPU "
                         "kernel at its real shape")
    ap.add_argument("--stream-sweep", action="store_true",
                    help="instead of the bench line: the in-place stream's rate over buffers "
                         "of 8 MB ... 4 GB on 256 and 1024 workgroups (one JSON line each), "
                         "which shows where the memory side stops caching the footprint")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (the "
                         "reference dispatch for scaling HBM byte counters) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes_read": n * 4, "calibrate_copy_bytes_written": n * 4}))
        return
    if args.map_sweep:
        map_sweep(args.cpu_budget)
        return
    if args.stream_sweep:
        import torch
        torch.cuda.set_device(0)
        for mb in (8, 16, 32, 64, 82, 100, 128, 192, 256, 384, 512, 1024, 4096):
            for grid in (256, 1024):
                r = stream_inplace(mb * 1000 * 1000, grid)
                print(json.dumps({"stream_inplace_MB": mb, **r}), flush=True)
        return
    if args.batch_map:
        batch_map_epoch(args.workload, args.steps, args.warmup)
        return
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only; --gpus {args.gpus} is not "
              "supported (the path would shard prototype rows across GPUs with one "
              "8-byte arg-min exchange per step, which is not built)", file=sys.stderr)
        sys.exit(2)

    import workloads

    cfg = workloads.WORKLOADS[args.workload]
    shard = None
    if args.shard > 1:
        base = cfg
        if base.units % args.shard:
            sys.exit(f"bench.py: --shard {args.shard} does not divide the {base.units} units")
        share = base.units // args.shard
        r = max(k for k in range(1, int(share ** 0.5) + 1) if share % k == 0)
        cfg = dataclasses.replace(base, name=f"{base.name}_shard{args.shard}", rows=r,
                                  cols=share // r)
        shard = {"of_workload": base.name, "gpus": args.shard, "units": share,
                 "map": f"{r}x{share // r}",
                 "note": "one GPU's share of the prototype rows, same samples, d and schedule; "
                         "the per-step arg-min exchange between GPUs is not built"}
    import torch
    torch.cuda.set_device(0)

    res, X, order = measure(cfg, args.input, args.steps, args.warmup)
    out = {
        "metric": "SOM train prototype*dim updates/sec + % of HBM/MALL roofline, 1 MI355X",
        "value": res.pop("value"),
        "unit": "proto*dim updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": res.pop("config"),
    }
    out.update(res)
    if shard:
        out["config"]["shard"] = shard
    if args.cpu_budget > 0:
        host = host_cpu()
        out["cpu_baseline"] = cpu_baseline(cfg, X, order, args.cpu_budget)
        out["cpu_baseline"]["host"] = host
        # the same oracle on one core (a third of the budget), for the
        # single-core speed-up
        out["cpu_baseline_1core"] = cpu_baseline(cfg, X, order, args.cpu_budget / 3, threads=1)
    del X, order
    also = [int(t) for t in args.also.split(",") if t.strip()] if not shard else []
    if also:
        out["also"] = {}
        for wi in also:
            if wi == args.workload:
                continue
            c = workloads.WORKLOADS[wi]
            r, Xa, _ = measure(c, args.input, args.also_steps, 1)
            out["also"][c.name] = r
            del Xa
    print(json.dumps(out), flush=True)


def measure(cfg, input_kind: str, steps: int, warmup: int):
    """Time `steps` bench steps of one workload (after `warmup`); returns
    (result fields, X, order)."""
    import numpy as np
    import torch

    import paper_1905_09598_amd as som
    import workloads

    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)
    Xd = torch.from_numpy(X).cuda()
    od = torch.from_numpy(order).cuda()
    m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=cfg.init_seed)
    W0 = m.weights.clone()
    plan = m.plan()
    stream = torch.cuda.current_stream()
    sparse = input_kind == "csr"
    if sparse:
        # CSR form of the same rows (host-side input preparation, untimed)
        nz = X != 0
        indptr = np.zeros(cfg.n + 1, np.int64)
        np.cumsum(nz.sum(1), out=indptr[1:])
        r, c = np.nonzero(nz)
        csr = (torch.from_numpy(indptr).cuda(), torch.from_numpy(c.astype(np.int32)).cuda(),
               torch.from_numpy(X[r, c]).cuda())
        nnz_row = np.diff(indptr)
        # per step: the sample's non-zeros, gathered and scattered in fp64 for
        # every unit of the 64-unit workgroups
        sparse_bytes = float(nnz_row[order].sum()) * 2 * 8 * (-(-cfg.units // 64) * 64)

    def one_step(ev=None):
        m.weights = W0
        if ev is not None:
            ev[0].record(stream)
        if sparse:
            m.train_csr(*csr, cfg.epochs, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1, order=od)
        else:
            m.train(Xd, cfg.epochs, cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1, order=od)
        if ev is not None:
            ev[1].record(stream)
        # every sample's BMU, QE and TE from one batched BMU search
        return m.evaluate(Xd)

    for _ in range(warmup):
        one_step()
    torch.cuda.synchronize()

    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        _, qe, te = one_step(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    train_ms = [a.elapsed_time(b) for a, b in events]

    # Batched BMU (the evaluation's dense contraction X W^T on fp32 MFMA):
    # som_bmu over all n samples, timed with HIP events on the same stream.
    bmu_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(3)]
    for a, b in bmu_ev:
        a.record(stream)
        m.bmu(Xd)
        b.record(stream)
    torch.cuda.synchronize()
    bmu_s = min(a.elapsed_time(b) for a, b in bmu_ev) / 1e3
    bmu_flops = 2.0 * cfg.n * cfg.units * cfg.d
    avg_train_s = sum(train_ms) / len(train_ms) / 1e3
    updates = cfg.steps * cfg.units * cfg.d
    ms_per_step = wall / steps * 1e3
    alg_bytes = cfg.steps * 3.0 * cfg.units * cfg.d * 4
    achieved = alg_bytes / avg_train_s / 1e9
    traffic = measured_traffic(cfg.name)
    kernel_name = ["train_kernel (stream)", "train_kernel (lds)",
                   "train_pipe_kernel (stream)", "train_pipe_kernel (lds)",
                   "train_pipe_kernel (stream, column walk)"][plan["variant"]]
    variant = ["stream", "lds", "pipelined-stream", "pipelined-lds",
               "pipelined-stream-cols"][plan["variant"]]
    grid, block = plan["grid"], plan["block"]
    # the LDS-resident kernels keep W on chip and wait on the grid exchange;
    # the streamed ones read and write W once per block of steps
    bound = "hbm" if plan["variant"] in (0, 2, 4) else "latency"
    if sparse:
        # the sparse path's own bytes: the dense 3 N d 4 per step does not
        # describe a kernel that touches only the sample's features
        alg_bytes = sparse_bytes
        achieved = alg_bytes / avg_train_s / 1e9
        traffic = None
        kernel_name = "sparse_train_kernel"
        variant = "csr lazy-scale"
        grid, block = -(-cfg.units // 64), 128
        bound = "latency"
    ref = stream_inplace(cfg.units * cfg.d * 4, grid if not sparse else 256)
    roof = {
        "bound": bound,
        "achieved": achieved,
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": achieved / HBM_PEAK_GBS,
        # the same algorithmic-byte rate under its own name: a figure of the
        # 3 N d 4 byte model, not of memory use (frac_applicable is that)
        "metric_frac": achieved / HBM_PEAK_GBS,
        "traffic": traffic,
        "kernel": kernel_name,
        "kernel_ms": avg_train_s * 1e3,
        "alg_bytes_per_launch": alg_bytes,
        "stream_inplace": ref,
    }
    if traffic:
        phys = traffic / avg_train_s / 1e9
        roof["traffic_source"] = ("FETCH_SIZE + WRITE_SIZE of this kernel source on this "
                                  "workload, stored in profiles/train_kernel_traffic.json")
        roof["traffic_GBs"] = phys
        roof["frac_hbm_traffic"] = phys / HBM_PEAK_GBS
        roof["frac_applicable"] = phys / ref["GB/s"]
    if sparse:
        roof["note"] = ("sparse path: bytes = the samples' non-zeros gathered and scattered in "
                        "fp64 for every unit; its step is bound by the grid exchange's latency, "
                        "not by bytes")
    res = {
        "value": updates / (ms_per_step / 1e3),
        "ms_per_step": ms_per_step,
        "config": {
            "workload": cfg.name, "n": cfg.n, "d": cfg.d,
            "map": f"{cfg.rows}x{cfg.cols}", "epochs": cfg.epochs,
            "train_steps_per_pass": cfg.steps,
            "schedule": f"lr {cfg.lr0}->{cfg.lr1} linear, sigma {cfg.sigma0}->{cfg.sigma1} exp",
            "grid": grid, "block": block, "variant": variant, "input": input_kind,
            "block_steps": None if sparse else plan["block_steps"],
        },
        "roofline": roof,
        "bmu_mfma": {
            "achieved": bmu_flops / bmu_s / 1e12, "peak": FP32_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": bmu_flops / bmu_s / 1e12 / FP32_MFMA_PEAK_TFLOPS,
            "flops": bmu_flops, "ms": bmu_s * 1e3,
            "note": "som_bmu over all n samples: 2 n N d flops of X W^T (fp32 MFMA) plus "
                    "the candidate re-rank, best of 3",
        },
        "train_ms": avg_train_s * 1e3,
        "us_per_sample_step": avg_train_s / cfg.steps * 1e6,
        "qe": qe,
        "te": te,
    }
    m.close()
    del Xd, od, W0
    torch.cuda.empty_cache()
    return res, X, order


if __name__ == "__main__":
    main()
