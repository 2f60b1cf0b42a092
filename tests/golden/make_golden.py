"""Write the end-to-end expected values of one training workload.

Calls only the fp64 oracle and the seeded input generators: it trains the
oracle over the workload's full schedule from its seeded initial map and
records the final quantization and topographic errors, together with
checksums of every input so that a test can prove it trains on the same
bits.

    python tests/golden/make_golden.py CONFIG_INDEX [--threads T] [--topology hex]

writes tests/golden/e2e_<config name>.json (e2e_<config name>_hex.json for
the hexagonal lattice).
"""
import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workloads  # noqa: E402


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("config", type=int)
    ap.add_argument("--threads", type=int, default=oracle.default_threads())
    ap.add_argument("--topology", choices=("rect", "hex"), default="rect")
    ap.add_argument("--out-dir", default=os.path.join(ROOT, "tests", "golden"),
                    help="directory of the record (default: tests/golden)")
    ap.add_argument("--epoch-qe", action="store_true",
                    help="also record the quantization error after every epoch")
    args = ap.parse_args()
    cfg = workloads.WORKLOADS[args.config]
    topo = oracle.HEX if args.topology == "hex" else oracle.RECT
    t0 = time.time()
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)
    W = oracle.init_uniform(cfg.init_seed, cfg.units, cfg.d)
    s = oracle.schedule(cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                        oracle.LINEAR, oracle.EXPONENTIAL)
    T = cfg.steps
    print(f"[golden] {cfg.name}: data {time.time() - t0:.1f}s, T={T}, "
          f"threads={args.threads}", flush=True)
    epoch_qe = []
    t1 = time.time()
    for e in range(cfg.epochs):
        sl = order[e * cfg.n:(e + 1) * cfg.n]
        W, _ = oracle.train(W, cfg.rows, cfg.cols, X, sl, s, step0=e * cfg.n,
                            total_steps=T, topology=topo, nthreads=args.threads)
        msg = f"[golden] {cfg.name}: epoch {e + 1}/{cfg.epochs} " \
              f"at {time.time() - t1:.0f}s"
        if args.epoch_qe:
            q = oracle.evaluate(W, cfg.rows, cfg.cols, X, topology=topo,
                                nthreads=args.threads)["qe"]
            epoch_qe.append(q)
            msg += f" qe={q:.6f}"
        print(msg, flush=True)
    train_s = time.time() - t1
    ev = oracle.evaluate(W, cfg.rows, cfg.cols, X, topology=topo, nthreads=args.threads)
    c1 = ev["c1"]
    rel_gap = np.where(ev["d1"] > 0, (ev["d2"] - ev["d1"]) / np.maximum(ev["d1"], 1e-300),
                       np.inf)
    out = {
        "written_by": "tests/golden/make_golden.py (fp64 oracle only)",
        "config": cfg.name,
        "n": cfg.n, "d": cfg.d, "rows": cfg.rows, "cols": cfg.cols,
        "epochs": cfg.epochs, "steps": T, "topology": args.topology,
        "schedule": {"lr0": cfg.lr0, "lr1": cfg.lr1, "lr_decay": "linear",
                     "sigma0": cfg.sigma0, "sigma1": cfg.sigma1,
                     "sigma_decay": "exponential"},
        "init_seed": cfg.init_seed, "shuffle_seed": cfg.shuffle_seed,
        "sha256_X": workloads.sha256_of(X),
        "sha256_order": workloads.sha256_of(order),
        "sha256_W0_f32": workloads.sha256_of(
            oracle.init_uniform(cfg.init_seed, cfg.units, cfg.d).astype(np.float32)),
        "qe": ev["qe"], "te": ev["te"],
        "te_count": int(round(ev["te"] * cfg.n)),
        "epoch_qe": epoch_qe,
        "units_used": int(np.unique(c1).size),
        "near_tie_samples_1e-4": int(np.sum(rel_gap <= 1e-4)),
        "oracle_train_seconds": round(train_s, 1),
        "oracle_threads": args.threads,
        "host": platform.processor() or platform.machine(),
    }
    suffix = "_hex" if args.topology == "hex" else ""
    os.makedirs(args.out_dir, exist_ok=True)
    path = os.path.join(args.out_dir, f"e2e_{cfg.name}{suffix}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(f"[golden] wrote {path}: qe={ev['qe']:.6f} te={ev['te']:.6f} "
          f"train {train_s:.0f}s", flush=True)


if __name__ == "__main__":
    main()
