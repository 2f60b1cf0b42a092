"""Measure how far the fp64 oracle's own end-of-training QE and TE move
between equally valid trainings of one workload.

Calls only the fp64 oracle and the seeded input generators.  Training k
(k = 1, 2, ...) runs the workload's full schedule on the same samples, the
same sample order and the same initial map as the stored end-to-end run,
with the oracle's own steps, except that every near tie -- a step whose two
smallest distances differ by at most TIE_REL of the smaller -- is decided
by a coin seeded with k (oracle.train_near_tie).  TIE_REL = 1e-6 is about
sixteen fp32 units in the last place: two distances that close cannot be
told apart by a distance summed in fp32 over hundreds to thousands of
terms, so every such training is as valid as the stored one, and the spread
of their QE and TE is the drift that runs of this precision show once they
part at a near tie.  (Moving the initial map or the state by one fp32 ulp
does not do this: the steps contract such a difference below the gaps of
the near ties, and those runs end with the stored TE.)

    python tests/golden/make_te_spread.py CONFIG_INDEX --runs K [--first k0]
        [--threads T] [--topology hex]

appends runs k0 .. k0+K-1 to te_spread_<config name>.json in --out-dir
(default tests/golden)
(..._hex.json for the hexagonal lattice), one record per finished training,
so an interrupted series keeps what it finished.
"""
import argparse
import fcntl
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


TIE_REL = 1e-6


def record(path: str, entry: dict, header: dict) -> None:
    with open(path, "a+") as f:
        fcntl.flock(f, fcntl.LOCK_EX)
        f.seek(0)
        text = f.read()
        doc = json.loads(text) if text.strip() else dict(header, runs=[])
        doc["runs"] = [r for r in doc["runs"] if r["k"] != entry["k"]] + [entry]
        doc["runs"].sort(key=lambda r: r["k"])
        f.seek(0)
        f.truncate()
        json.dump(doc, f, indent=1)
        f.write("\n")
        fcntl.flock(f, fcntl.LOCK_UN)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("config", type=int)
    ap.add_argument("--runs", type=int, default=1)
    ap.add_argument("--first", type=int, default=1)
    ap.add_argument("--threads", type=int, default=oracle.default_threads())
    ap.add_argument("--topology", choices=("rect", "hex"), default="rect")
    ap.add_argument("--out-dir", default=os.path.join(ROOT, "tests", "golden"),
                    help="directory of the record (default: tests/golden)")
    args = ap.parse_args()
    cfg = workloads.WORKLOADS[args.config]
    topo = oracle.HEX if args.topology == "hex" else oracle.RECT
    X = workloads.make_data(cfg)
    order = workloads.epoch_orders(cfg.n, cfg.epochs, cfg.shuffle_seed)
    s = oracle.schedule(cfg.lr0, cfg.lr1, cfg.sigma0, cfg.sigma1,
                        oracle.LINEAR, oracle.EXPONENTIAL)
    suffix = "_hex" if args.topology == "hex" else ""
    os.makedirs(args.out_dir, exist_ok=True)
    path = os.path.join(args.out_dir, f"te_spread_{cfg.name}{suffix}.json")
    header = {
        "written_by": "tests/golden/make_te_spread.py (fp64 oracle only)",
        "config": cfg.name, "n": cfg.n, "topology": args.topology,
        "near_tie": f"D2 - D1 <= {TIE_REL} D1 decided by bit 63 of SplitMix64(1000 + k, step)",
        "sha256_X": workloads.sha256_of(X),
        "sha256_order": workloads.sha256_of(order),
    }
    W0 = oracle.init_uniform(cfg.init_seed, cfg.units, cfg.d)
    for k in range(args.first, args.first + args.runs):
        W = W0
        flips = 0
        t0 = time.time()
        for e in range(cfg.epochs):
            sl = order[e * cfg.n:(e + 1) * cfg.n]
            W, f = oracle.train_near_tie(W, cfg.rows, cfg.cols, X, sl, s, TIE_REL, 1000 + k,
                                         step0=e * cfg.n, total_steps=cfg.steps,
                                         topology=topo, nthreads=args.threads)
            flips += f
            print(f"[spread] {cfg.name}{suffix} k={k}: epoch {e + 1}/{cfg.epochs} "
                  f"at {time.time() - t0:.0f}s, {flips} near ties flipped", flush=True)
        ev = oracle.evaluate(W, cfg.rows, cfg.cols, X, topology=topo,
                             nthreads=args.threads)
        entry = {"k": k, "qe": ev["qe"], "te": ev["te"],
                 "te_count": int(round(ev["te"] * cfg.n)),
                 "near_ties_flipped": flips,
                 "oracle_train_seconds": round(time.time() - t0, 1),
                 "oracle_threads": args.threads,
                 "host": platform.processor() or platform.machine()}
        record(path, entry, header)
        print(f"[spread] {cfg.name}{suffix} k={k}: qe={ev['qe']:.6f} "
              f"te_count={entry['te_count']}", flush=True)


if __name__ == "__main__":
    main()
