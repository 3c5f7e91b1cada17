"""Write the per-update losses of simultaneous (one-shot) layer-parallel training
on the one-shot workload (dense width 32, N = 1024, B = 16384, 3-level MGRIT
with one forward and one adjoint iteration per update, plain
gradient step lr = 1e-2; Algorithm 2 with m1 = m2 = 1 and a scaled-identity
Hessian approximation), next to layer-serial gradient descent from the same
seed, both computed by the fp64 oracle.

Only oracle/ and workloads/ are called. The oracle is slow at this size (minutes
per update), so the file holds the first one-shot updates and, optionally, as
many layer-serial updates. Usage:
    python tests/golden/make_one_shot_golden.py [one_shot_updates] [serial_updates]
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle as O  # noqa: E402
from workloads import ONE_SHOT_LR, ONE_SHOT_UPDATES, WORKLOADS, generate  # noqa: E402


def main():
    n_oneshot = int(sys.argv[1]) if len(sys.argv) > 1 else 10
    n_serial = int(sys.argv[2]) if len(sys.argv) > 2 else 0
    wl = WORKLOADS[5]
    d = generate(wl)
    args = (d["y"], d["onehot"], d["L_in"], d["K"], d["b"], d["W"], d["mu"], wl.h, wl.act, wl.opening)
    t0 = time.time()
    lo, _ = O.one_shot(*args, cf=wl.cf, max_levels=wl.max_levels, min_coarse=wl.min_coarse, relax=wl.relax,
                       updates=n_oneshot, lr=ONE_SHOT_LR, m1=wl.fwd_iters, m2=wl.adj_iters)
    t1 = time.time()
    print(f"one-shot: {n_oneshot} updates in {t1 - t0:.0f} s", file=sys.stderr, flush=True)
    ls, _ = O.serial_training(*args, updates=n_serial, lr=ONE_SHOT_LR) if n_serial else ([], None)
    t2 = time.time()
    out = os.path.join(HERE, "one_shot_losses.txt")
    with open(out, "w") as f:
        f.write("# Losses of the one-shot workload (dense tanh, width 32, N = 1024, B = 16384, seeds 1005/2005),\n")
        f.write(f"# plain gradient steps, lr = {ONE_SHOT_LR}; fp64 oracle on the fp32-rounded inputs.\n")
        f.write("# Written by tests/golden/make_one_shot_golden.py (calls oracle/ only).\n")
        f.write("# columns: update  one-shot loss (1 forward + 1 adjoint MGRIT iteration)  layer-serial\n")
        f.write("# loss (nan past the computed updates)\n")
        for i in range(max(len(lo), len(ls))):
            a = lo[i] if i < len(lo) else float("nan")
            b = ls[i] if i < len(ls) else float("nan")
            f.write(f"{i} {a:.17g} {b:.17g}\n")
    print(f"wrote {out}: one-shot {t1 - t0:.0f} s, serial {t2 - t1:.0f} s")


if __name__ == "__main__":
    main()
