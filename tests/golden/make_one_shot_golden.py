"""Write the per-update losses of simultaneous (one-shot) layer-parallel training
on the one-shot workload (dense width 32, N = 1024, B = 16384, 3-level MGRIT
with one forward and one adjoint iteration per update, plain
gradient step lr = 1e-2; Algorithm 2 with m1 = m2 = 1 and a scaled-identity
Hessian approximation), next to layer-serial gradient descent from the same
seed (exact forward propagation and backpropagation), both computed by the
fp64 oracle.

Only oracle/ and workloads/ are called. The oracle is slow at this size (about
two minutes per one-shot update on one core), so the two runs go to two
processes, and each appends its losses to a partial file as they come
(`one_shot_losses.<run>.part`), so an interrupted run keeps what it finished;
the final table is assembled from the partial files. Usage:

    python tests/golden/make_one_shot_golden.py [one_shot_updates] [serial_updates]
    python tests/golden/make_one_shot_golden.py --assemble   # table from the partial files
"""
import multiprocessing as mp
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle as O  # noqa: E402
from workloads import ONE_SHOT_LR, ONE_SHOT_UPDATES, WORKLOADS, generate  # noqa: E402

OUT = os.path.join(HERE, "one_shot_losses.txt")


def part_path(run):
    return os.path.join(HERE, f"one_shot_losses.{run}.part")


def run(kind, updates):
    wl = WORKLOADS[5]
    d = generate(wl)
    args = (d["y"], d["onehot"], d["L_in"], d["K"], d["b"], d["W"], d["mu"], wl.h, wl.act, wl.opening)
    path = part_path(kind)
    t0 = time.time()
    with open(path, "w") as f:
        def progress(it, J):
            f.write(f"{it} {J:.17g}\n")
            f.flush()
            print(f"[{kind}] update {it} J={J:.10f} ({time.time() - t0:.0f} s)", file=sys.stderr, flush=True)

        if kind == "oneshot":
            O.one_shot(*args, cf=wl.cf, max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=wl.relax,
                       updates=updates, lr=ONE_SHOT_LR, m1=wl.fwd_iters, m2=wl.adj_iters, progress=progress)
        else:
            O.serial_training(*args, updates=updates, lr=ONE_SHOT_LR, progress=progress)


def read_part(kind):
    path = part_path(kind)
    if not os.path.exists(path):
        return []
    vals = []
    for line in open(path):
        i, v = line.split()
        assert int(i) == len(vals), path
        vals.append(float(v))
    return vals


def assemble():
    lo, ls = read_part("oneshot"), read_part("serial")
    with open(OUT, "w") as f:
        f.write("# Losses of the one-shot workload (dense tanh, width 32, N = 1024, B = 16384, seeds 1005/2005),\n")
        f.write(f"# plain gradient steps, lr = {ONE_SHOT_LR}; fp64 oracle on the fp32-rounded inputs.\n")
        f.write("# Written by tests/golden/make_one_shot_golden.py (calls oracle/ only).\n")
        f.write("# columns: update  one-shot loss (1 forward + 1 adjoint MGRIT iteration)  layer-serial\n")
        f.write("# loss (exact forward propagation + backpropagation; nan past the computed updates)\n")
        for i in range(max(len(lo), len(ls))):
            a = lo[i] if i < len(lo) else float("nan")
            b = ls[i] if i < len(ls) else float("nan")
            f.write(f"{i} {a:.17g} {b:.17g}\n")
    print(f"wrote {OUT}: {len(lo)} one-shot and {len(ls)} layer-serial updates")


def main():
    if len(sys.argv) > 1 and sys.argv[1] == "--assemble":
        assemble()
        return
    n_oneshot = int(sys.argv[1]) if len(sys.argv) > 1 else ONE_SHOT_UPDATES
    n_serial = int(sys.argv[2]) if len(sys.argv) > 2 else ONE_SHOT_UPDATES
    procs = [mp.Process(target=run, args=(k, n)) for k, n in (("oneshot", n_oneshot), ("serial", n_serial)) if n]
    for p in procs:
        p.start()
    for p in procs:
        p.join()
    if any(p.exitcode for p in procs):
        raise SystemExit("an oracle run failed")
    assemble()


if __name__ == "__main__":
    main()
