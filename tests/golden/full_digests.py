"""Checksums of every output on every block index of the full-size workloads,
computed with the oracle (and the host input generator) only; the GPU parity
tests compute the same checksums of the GPU's outputs on the device
(tests/digest.py defines the streams and the checksum).

With one team (d = 1), and within the teams' block numbering for R-SAG and
B-SAG, block b of every output depends only on block b of every worker's
inputs over all steps, so each block index is an independent job: its
residual is carried from step to step like the GPU's.

    python tests/golden/full_digests.py --workload 3 --form eager --jobs 4
    python tests/golden/full_digests.py --workload 2 --form bsag --teams 4

writes tests/golden/digests_w<workload>_<form>[_d<teams>].json.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def out_path(workload: int, form: str, d: int = 1) -> str:
    suffix = f"_d{d}" if form in ("rsag", "bsag") else ""
    return os.path.join(HERE, f"digests_w{workload}_{form}{suffix}.json")


def team_sizes(wl, d: int):
    """Blocks per team and L = d k / P of the team variants (k = P k_blk)."""
    return wl.P // d, d * wl.k_blk


def block_job(args) -> tuple:
    workload, form, d, b = args
    from oracle import spardl_oracle as so
    from paper_2304_00737_amd import workloads as W
    from tests.digest import host_digest, host_streams

    wl = W.config(workload)
    P, n, kb = wl.P, wl.n, wl.k_blk
    nb, L = (P, kb) if form in ("eager", "lazy") else team_sizes(wl, d)
    bounds = so.block_bounds(n, nb)
    lo, hi = bounds[b], bounds[b + 1]
    acc = [{b: np.zeros(hi - lo, np.float32)} for _ in range(P)]
    ctrl = {}
    bags = [len(s.received_bag[0]) for s in so.srs_schedule(nb)]
    steps = []
    t0 = time.time()
    for t in range(1, wl.steps + 1):
        grad = []
        for w in range(P):
            h = np.empty(hi - lo, np.float32)
            W.fill(h, wl, t, w, x0=lo)
            grad.append({b: h})
        if form == "eager":
            res = so.spardl_step(acc, grad, P, n, kb, blocks=[b])
        elif form == "lazy":
            res = so.spardl_step_lazy(acc, grad, P, n, kb, blocks=[b])
        elif form == "rsag":
            res = so.spardl_step_rsag(acc, grad, P, n, L, d, blocks=[b])
        else:
            res = so.spardl_step_bsag(acc, grad, P, n, L, d, ctrl, blocks=[b])
        steps.append(host_digest(host_streams(form, res, P, b, bags, Q=nb, d=d, steps=d.bit_length() - 1, L=L)))
        del res, grad
    return b, steps, time.time() - t0


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", type=int, required=True)
    ap.add_argument("--form", choices=("eager", "lazy", "rsag", "bsag"), default="eager")
    ap.add_argument("--teams", type=int, default=1)
    ap.add_argument("--jobs", type=int, default=1)
    ap.add_argument("--blocks", type=str, default="", help="comma-separated block indices (default: all)")
    args = ap.parse_args()
    from oracle import spardl_oracle as so
    from paper_2304_00737_amd import workloads as W

    wl = W.config(args.workload)
    d = args.teams if args.form in ("rsag", "bsag") else 1
    nb = wl.P if d == 1 else wl.P // d
    blocks = [int(x) for x in args.blocks.split(",")] if args.blocks else list(range(nb))
    path = out_path(args.workload, args.form, d)
    out = {"workload": wl.name, "form": args.form, "teams": d, "P": wl.P, "n": wl.n, "k_per_block": wl.k_blk,
           "blocks_per_row": nb, "steps": wl.steps, "bounds": [int(x) for x in so.block_bounds(wl.n, nb)],
           "digests": {}}
    if os.path.exists(path):   # resume: keep block indices already done
        old = json.load(open(path))
        if all(old.get(k) == out[k] for k in ("workload", "form", "teams", "P", "n", "steps")):
            out["digests"] = old["digests"]
    todo = [b for b in blocks if str(b) not in out["digests"]]
    print(f"{wl.name} {args.form} d={d}: {len(todo)} block indices to do, {args.jobs} jobs", flush=True)
    with ProcessPoolExecutor(max_workers=args.jobs) as ex:
        for b, steps, secs in ex.map(block_job, [(args.workload, args.form, d, b) for b in todo]):
            out["digests"][str(b)] = steps
            with open(path + ".tmp", "w") as f:
                json.dump(out, f, indent=0)
            os.replace(path + ".tmp", path)
            print(f"block {b}: {secs:.0f} s", flush=True)
    print("wrote", path)


if __name__ == "__main__":
    main()
