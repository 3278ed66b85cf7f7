"""Throughput of one full SparDL synchronisation step (d = 1) on one MI355X.

A step is the whole hot path for P simulated workers over one batch of
gradients: residual add (fused level-1 histogram and speculative
candidates), block top-k/P, the ceil(log2 P) Spar-Reduce-Scatter steps, the
All-Gather decode to a dense update, and global residual collection.

The line's `value` is the ResNet-50-sized workload: P = 8, n = 25.6M fp32
per worker, density 1%, three distinct gradient batches cycled with the
residual carried across steps, inputs resident in HBM before timing starts.
The default run then adds two sub-objects: the GPT-2-XL-sized workload
(P = 32, n = 1.5e9, 0.1%; its residual alone is 192 GB, so each worker's
gradient is generated on the GPU between that worker's calls, untimed) and
the launch-bound P = 4, n = 2^20 workload replayed from a captured HIP graph
beside eager launches.  Before any GPU work, the oracle is timed on the
host's cores on whole block indices of the headline workload.

Prints one JSON line (see the "metric" field); timing uses HIP events on the
stream the kernels run on.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E peak, GB/s
CALIB_BYTES = 1 << 30   # bytes read (and written) by the calibration copy


def _kernel_src_hash() -> str:
    """Hash of the residual-add kernel's source (its file, with its launcher,
    and the headers it includes), to tell whether stored counter readings
    still describe the kernel being timed."""
    csrc = os.path.join(ROOT, "paper_2304_00737_amd", "csrc")
    h = hashlib.sha256()
    for f in ("kernels_add.hip", "device.hpp", "common.hpp"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _traffic_from_profiles(kernel: str, src_hash: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source and on this workload; otherwise None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    k = rec.get("kernels", {}).get(kernel)
    if not k or rec.get("src_hash") != src_hash or rec.get("workload") != workload:
        return None
    return k.get("bytes_per_launch")


def _oracle_block(job):
    """One block index of a workload through all its steps with the residual
    carried (blocks never interact, so this is a self-contained unit):
    returns (gradient elements processed, seconds inside the oracle)."""
    cfg, lazy, b = job
    import numpy as np

    from oracle import spardl_oracle as so
    from paper_2304_00737_amd import workloads as W

    wl = W.config(cfg)
    P, n, kb = wl.P, wl.n, wl.k_blk
    bounds = so.block_bounds(n, P)
    step_fn = so.spardl_step_lazy if lazy else so.spardl_step
    acc = [{b: np.zeros(bounds[b + 1] - bounds[b], np.float32)} for _ in range(P)]
    secs, elems = 0.0, 0
    for t in range(1, wl.steps + 1):
        grad = [{b: W.gradient(wl, t, w, bounds[b], bounds[b + 1] - bounds[b])} for w in range(P)]
        t0 = time.perf_counter()
        step_fn(acc, grad, P, n, kb, blocks=[b])
        secs += time.perf_counter() - t0
        elems += P * (bounds[b + 1] - bounds[b])
    return elems, secs


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# worker processes of the oracle baseline: the host's cores, but no more than
# the CPU share of one GPU on a shared node
CPU_SHARE = 16


def cpu_baseline(wl, lazy: bool = False):
    """The oracle, as it stands, on the headline workload: every block index
    (a self-contained unit of a step) through the workload's steps with its
    residual carried, one block index per worker process, all at once, on
    every core of the host's share (block indices repeat when there are more
    cores than block indices, so that no core idles); plus block index 0
    alone in one process (the single-thread figure).  Runs before anything
    touches the GPU; worker processes are started fresh (spawn), not
    forked."""
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor

    P = wl.P
    nproc = os.cpu_count() or 1
    procs = max(1, min(nproc, CPU_SHARE))
    jobs = [b % P for b in range(max(procs, P))]   # every block index, then repeats for the spare cores
    e1, s1 = _oracle_block((wl.cfg_id, lazy, 0))
    t0 = time.perf_counter()
    with ProcessPoolExecutor(max_workers=procs, mp_context=mp.get_context("spawn")) as ex:
        res = list(ex.map(_oracle_block, [(wl.cfg_id, lazy, b) for b in jobs]))
    wall = time.perf_counter() - t0
    elems = sum(e for e, _ in res)
    # oracle time only, as for the single-thread figure: the processes run their block indices
    # concurrently, so the pool takes as long as its slowest process
    secs = max(max(x for _, x in res), sum(x for _, x in res) / procs)
    return {"value": elems / secs, "unit": "elements/s", "cores": procs, "kind": "oracle",
            "nproc": nproc, "cpu_model": _cpu_model(),
            "single_thread_value": e1 / s1,
            "sample": f"the whole workload: its {P} block indices x {wl.steps} steps with the residual carried, "
                      f"{len(jobs)} block-index jobs ({elems} gradient elements), one per process on {procs} "
                      f"processes at once: "
                      f"{secs:.1f} s inside the oracle for the slowest process ({wall:.1f} s wall with process "
                      f"start and input generation); single-thread figure: block index 0 alone ({e1} "
                      f"elements, {s1:.1f} s in the oracle; numpy)"}


def ws_check(st) -> None:
    from paper_2304_00737_amd import spardl
    for ws in [getattr(st, "ws", None), getattr(st, "ws_sag", None)] + list(getattr(st, "ws_team", [])):
        if ws is not None:
            assert spardl.ws_error(ws) == 0


def rsag_exchange(st, t: int) -> None:
    from paper_2304_00737_amd import spardl
    spardl.rsag_merge_topk(st.sp_idx, st.sp_val, st.P, st.d, st.n, st.k_blk, t, st.sag_idx[t], st.sag_val[t],
                           st.sag_cnt[t], st.ws_sag)


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=2, help="synthetic workload id (1-5)")
    ap.add_argument("--variant", choices=("eager", "lazy"), default="eager",
                    help="eager: re-select after every merge (the hot path); lazy: sparsify a block only "
                         "when it is sent (Sec. III-B, Optimization for SRS)")
    ap.add_argument("--teams", type=int, default=1,
                    help="d > 1: d teams of P/d workers joined by R-SAG (Sec. III-D; d a power of 2), "
                         "L = d k / P entries per team block")
    ap.add_argument("--bruck", action="store_true",
                    help="with --teams d: join the teams by B-SAG (any d dividing P; Algorithm 2 sets h)")
    ap.add_argument("--rows-per-call", type=int, default=0,
                    help="workload 5: workers per residual-add / block top-k call (default PER_WORKER_ROWS)")
    ap.add_argument("--separate-collect", action="store_true",
                    help="eager variant: run the global residual collection as its own call at the end of "
                         "each step (by default it runs inside the next step's residual add, which reads "
                         "and writes every element of the residual anyway)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the GPT-2-XL-sized and HIP-graph sub-objects of the default run")
    ap.add_argument("--w5-steps", type=int, default=2, help="timed steps of the GPT-2-XL-sized sub-object")
    ap.add_argument("--w5-warmup", type=int, default=1)
    ap.add_argument("--graph-steps", type=int, default=200, help="timed steps of the HIP-graph sub-object")
    ap.add_argument("--calib-copy", action="store_true",
                    help="first run one untimed device-to-device copy of CALIB_BYTES (a reference "
                         "kernel of known traffic for hardware-counter runs)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs the P simulated workers on one GPU; "
                                   "--gpus must be 1 (no multi-GPU path is built)"}))
        return 2

    from paper_2304_00737_amd import workloads as W

    wl = W.config(args.workload)
    # the oracle baseline first: its worker processes start before anything touches the GPU
    cpu_base = None
    if not args.no_cpu_baseline and args.teams == 1 and 4.0 * wl.P * wl.n * (wl.steps + 1) <= PER_WORKER_BYTES:
        cpu_base = cpu_baseline(wl, lazy=args.variant == "lazy")

    import numpy as np
    import torch

    from paper_2304_00737_amd import spardl

    P, n, kb = wl.P, wl.n, wl.k_blk
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lazy = args.variant == "lazy"
    d = args.teams
    if d > 1 and (lazy or P % d or (d & (d - 1) and not args.bruck)):
        print(json.dumps({"error": "--teams needs a d dividing P (a power of two without --bruck), "
                                   "with the eager variant"}))
        return 2
    if 4.0 * P * n * (wl.steps + 1) > PER_WORKER_BYTES:
        return run_per_worker(args, wl, dev)

    # inputs: the workload's distinct gradient batches, resident in HBM
    t0 = time.time()
    grads = []
    for t in range(1, wl.steps + 1):
        g = torch.empty((P, n), dtype=torch.float32, device=dev)
        host = np.empty(n, np.float32)
        for w in range(P):
            W.fill(host, wl, t, w)
            g[w].copy_(torch.from_numpy(host))
        grads.append(g)
    torch.cuda.synchronize()
    print(f"# generated {wl.steps} x {P} x {n} gradients in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    if args.calib_copy:
        src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    stream = torch.cuda.current_stream()
    if d > 1:
        L = d * wl.k_blk
        st = spardl.SparDLSagStep(P, d, n, L, device=dev, bruck=args.bruck)
        if args.bruck:
            calls = ["add_and_block_topk", "team_srs", "bsag_exchange", "allgather_densify", "residual_collect"]

            def call_fns(j):
                g = grads[j % len(grads)]
                return [lambda: st.add_and_select(g), st.team_srs, st.exchanges, st.densify, st.collect]
        else:
            calls = ["add_and_block_topk", "team_srs"] + [f"exchange{t}" for t in range(st.steps)] + \
                    ["allgather_densify", "residual_collect"]

            def call_fns(j):
                g = grads[j % len(grads)]
                return [lambda: st.add_and_select(g), st.team_srs] + \
                       [(lambda t=t: rsag_exchange(st, t)) for t in range(st.steps)] + [st.densify, st.collect]
    elif lazy:
        st = spardl.SparDLLazyStep(P, n, kb, device=dev)
        calls = ["residual_add"] + [c for i in range(1, st.l + 1) for c in (f"topk_step{i}", f"receive_step{i}")] + \
                ["topk_reserved", "allgather_densify", "residual_collect"]

        def call_fns(j):
            g = grads[j % len(grads)]
            fns = [lambda: st.residual_add_rows(0, g)]
            for i in range(1, st.l + 1):
                fns += [lambda i=i: st.topk_round(i), lambda i=i: st.receive(i)]
            return fns + [lambda: st.topk_round(0), st.densify, st.collect]
    else:
        st = spardl.SparDLStep(P, n, kb, device=dev, fuse_collect=not args.separate_collect)
        calls = ["residual_add", "block_topk"] + [f"merge_step{i}" for i in range(1, st.l + 1)] + \
                ["allgather_densify", "residual_collect"]

        def call_fns(j):
            g = grads[j % len(grads)]
            return [lambda: st.residual_add(g), st.block_topk] + \
                   [(lambda i=i: st.merge_round(i)) for i in range(1, st.l + 1)] + [st.densify, st.collect]

    def ev():
        return torch.cuda.Event(enable_timing=True)

    for j in range(args.warmup):
        for f in call_fns(j):
            f()
    torch.cuda.synchronize()
    ws_check(st)

    # ---- timed region: K whole steps, one event pair around them
    start, end = ev(), ev()
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for j in range(args.steps):
        for f in call_fns(args.warmup + j):
            f()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ws_check(st)
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps
    dc = [] if lazy or d > 1 else [t.cpu().numpy() for t in st.drop_cnt]   # drops of the last timed step
    # the last timed step's speculative candidates and the blocks the top-k read again
    stats = spardl.topk_stats(st.ws, P, P, n, kb) if not lazy and d == 1 else None

    # ---- per-call attribution (untimed for `value`): events around every call.
    # An event record costs a fixed marker overhead on the stream; it is
    # measured with empty event pairs and subtracted.
    j0 = args.warmup + args.steps
    evs = [[(ev(), ev()) for _ in calls] for _ in range(args.steps)]
    empty = [(ev(), ev()) for _ in range(args.steps)]
    for j in range(args.steps):
        for c, f in enumerate(call_fns(j0 + j)):
            evs[j][c][0].record(stream)
            f()
            evs[j][c][1].record(stream)
        empty[j][0].record(stream)
        empty[j][1].record(stream)
    torch.cuda.synchronize()
    ws_check(st)
    marker_ms = sum(a.elapsed_time(b) for a, b in empty) / args.steps
    per_call_ms = {c: max(sum(evs[j][ci][0].elapsed_time(evs[j][ci][1]) for j in range(args.steps))
                          / args.steps - marker_ms, 0.0) for ci, c in enumerate(calls)}

    # ---- dominant kernel: the residual add is one kernel per call (with the
    # previous step's collection fused in; its drop index is built by the
    # collect call); each launch is bracketed by an event pair on its stream
    # (marker cost removed)
    g0 = grads[0]
    k_mid = [(ev(), ev()) for _ in range(args.steps)]
    for j in range(args.steps):
        k_mid[j][0].record(stream)
        if d > 1:
            st.add_and_select(g0)
            k_mid[j][1].record(stream)
        elif lazy:
            st.residual_add_rows(0, g0)
            k_mid[j][1].record(stream)
        else:
            st.residual_add(g0)
            k_mid[j][1].record(stream)
            st.block_topk()
            if st.fuse_collect:
                st.finish()   # the next add takes this step's collection, as in the timed steps
    torch.cuda.synchronize()
    add_ms = sum(a.elapsed_time(b) for a, b in k_mid) / args.steps - marker_ms
    ws_check(st)
    # the same rows through the plain residual add (no histogram, no candidates): the
    # streaming ceiling of this access pattern, beside the fused kernel; run on the
    # workspace's copy of acc so the step's state is untouched (g0 and -g0 alternate)
    plain_ms = None
    if d == 1 and not lazy:
        scratch_acc = st.acc.clone()
        neg = -g0
        pm = [(ev(), ev()) for _ in range(args.steps)]
        for j in range(args.steps):
            pm[j][0].record(stream)
            spardl.residual_add(scratch_acc, g0 if j % 2 == 0 else neg, P, n, 0, None)
            pm[j][1].record(stream)
        torch.cuda.synchronize()
        plain_ms = sum(a.elapsed_time(b) for a, b in pm) / args.steps - marker_ms
        del scratch_acc, neg
        torch.cuda.empty_cache()

    elems = P * n
    value = elems / (ms_per_step * 1e-3)

    # algorithmic HBM bytes per call (values and indices are 4 bytes)
    pairs = [P * m for m in st.bags]
    alg = {
        "residual_add": 12.0 * P * n,                              # read G, read xi, write A
        "allgather_densify": 4.0 * n + n / 8.0 + 8.0 * P * kb,     # write u and the bitmap of I; read the final blocks
    }
    if d > 1:
        Q, L = st.Q, st.k_blk
        alg["add_and_block_topk"] = 16.0 * P * n + 12.0 * P * Q * L
        alg["team_srs"] = sum(32.0 * P * m * L for m in st.bags)
        if args.bruck:
            # read every held block; write top-h and drops; the union reads the kept lists, writes and
            # reads the scatter row and writes the sums; the final selection reads them and writes sp
            alg["bsag_exchange"] = 16.0 * P * L + 8.0 * P * L + 16.0 * d * Q * L
            alg["allgather_densify"] = 4.0 * n + n / 8.0 + 8.0 * Q * L
            alg["residual_collect"] = 4.0 * P * Q * L + 8.0 * (P * Q * L) + 16.0 * P * L
        else:
            for t in range(st.steps):
                alg[f"exchange{t}"] = 40.0 * (d // 2) * Q * L     # read both blocks; write both kept + the drops
            alg["allgather_densify"] = 4.0 * n + n / 8.0 + 8.0 * Q * L
            alg["residual_collect"] = 4.0 * P * Q * L + 8.0 * (P * Q * L) + 24.0 * st.steps * (d // 2) * Q * L
        del alg["residual_add"]
    elif lazy:
        blk = n / P
        for i, pc in enumerate(pairs, start=1):
            alg[f"topk_step{i}"] = 4.0 * pc * blk + 8.0 * pc * kb  # read the sent blocks; write idx, val
            alg[f"receive_step{i}"] = 20.0 * pc * kb               # read idx, val; read, save and write acc
        alg["topk_reserved"] = 4.0 * P * blk + 8.0 * P * kb
        # read every selection; zero the selected final entries (upper bound: all); restore the
        # received entries off I (read idx and saved value, write; upper bound: all)
        alg["residual_collect"] = 8.0 * P * P * kb + 12.0 * sum(pairs) * kb
    else:
        alg["block_topk"] = 4.0 * P * n + 12.0 * P * P * kb        # read A; write idx, val, local idx
        for i, pc in enumerate(pairs, start=1):
            alg[f"merge_step{i}"] = 32.0 * pc * kb                 # read held + received, write kept + dropped
        drops_total = float(sum(int(d.sum()) for d in dc))
        # read local idx and drop lists; read+write touched residual entries (upper bound); the
        # membership lookups hit the bitmap of I that densify wrote (n/8 bytes, cache resident)
        alg["residual_collect"] = 4.0 * P * P * kb + 8.0 * drops_total + 8.0 * (P * P * kb + drops_total)
    # bytes the fused design moves (the headline step fraction): the add's stream plus the
    # candidates it writes; the top-k reads the candidates (and a block again only where it fell
    # back) and writes the selections.  The unfused figure prices the top-k at one more read of A
    # per element instead (16 B per gradient element): a labelled comparison only.
    moved = dict(alg)
    cand, reread = 0, 0
    if stats is not None:
        blen = [((b + 1) * n) // P - (b * n) // P for b in range(P)]
        cand = sum(stats["candidates"])
        reread = sum(blen[u % P] for u, ok in enumerate(stats["spec_ok"]) if not ok)
        moved["residual_add"] = 12.0 * P * n + 8.0 * cand
        moved["block_topk"] = 8.0 * cand + 4.0 * reread + 12.0 * P * P * kb
    dominant = max(calls, key=lambda c: per_call_ms[c])
    dom_ms = add_ms if dominant in ("residual_add", "add_and_block_topk") else per_call_ms[dominant]
    achieved = alg[dominant] / (dom_ms * 1e-3) / 1e9
    src_hash = _kernel_src_hash()
    # the stored counter readings are of the fused add (eager variant)
    traffic = None if lazy or d > 1 else _traffic_from_profiles(dominant, src_hash, wl.name)
    core_bytes = sum(v for k, v in alg.items() if k != "allgather_densify")
    full_bytes = sum(alg.values())

    out = {
        "metric": (f"gradient elements/sec per full SparDL step, {'B' if args.bruck else 'R'}-SAG with d={d} teams "
                   f"(P=8 virtual); % of HBM peak"
                   if d > 1 else
                   "gradient elements/sec per full SparDL step, lazy sparsification (P=8 virtual); % of HBM peak"
                   if lazy else "gradient elements/sec per full SparDL step (P=8 virtual); % of HBM peak"),
        "value": value,
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "P": P, "n_per_worker": n, "density": f"{wl.density[0]}/{wl.density[1]}",
                   "k_per_block": kb, "gradient_batches": wl.steps, "residual": "carried across steps",
                   "segments": len(wl.seg_len), "seed": W.SEED_BASE, "variant": args.variant, "teams": d,
                   "team_join": ("B-SAG" if args.bruck else "R-SAG") if d > 1 else None,
                   "L_per_team_block": st.k_blk if d > 1 else None,
                   "residual_collection": ("inside the next step's residual add" if getattr(st, "fuse_collect", False)
                                           else "its own call at the end of the step")},
        "roofline": {"bound": "hbm", "kernel": (("k_residual_add4<true, true> (the previous step's collection fused in)"
                                                  if getattr(st, "fuse_collect", False) else "k_residual_add4<true, false>")
                                                 if dominant == "residual_add" else dominant),
                     "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "alg_bytes_per_launch": alg[dominant], "avg_launch_ms": dom_ms,
                     "plain_add_ms": plain_ms,
                     "plain_add_GBs": (12.0 * P * n / (plain_ms * 1e-3) / 1e9) if plain_ms else None},
        "step_roofline": _step_roofline(moved, alg, ms_per_step, cand, reread, stats),
        "per_call_ms": per_call_ms,
        "event_marker_ms": marker_ms,
        "wall_s_timed": wall,
        "kernel_src": src_hash,
    }
    if cpu_base is not None:
        out["cpu_baseline"] = cpu_base
    if not args.no_extra and args.workload == 2 and d == 1 and not lazy:
        del st, grads, g0
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        # (the GPT-2-XL-sized rows keep the separate collection: at 0.1 % density the fused add's
        # reads of the final-index bitmap, n/8 bytes per row, cost more than the scattered writes)
        w5 = per_worker_measure(W.config(5), dev, args.w5_steps, args.w5_warmup, PER_WORKER_ROWS, False, False)
        out["workload5"] = {k: w5[k] for k in ("metric", "value", "ms_per_step", "steps", "warmup", "config",
                                               "roofline", "step_roofline", "per_call_ms", "span_ms_per_step")}
        torch.cuda.empty_cache()
        out["workload1_graph"] = graph_measure(W.config(1), dev, args.graph_steps)
    print(json.dumps(out), flush=True)
    return 0


def _step_roofline(moved, alg, ms_per_step, cand, reread, stats) -> dict:
    """Step bytes against the step time: the bytes this design moves (headline), and the unfused
    16 B per gradient element figure beside it."""
    sec = ms_per_step * 1e-3
    mfull = sum(moved.values())
    mcore = sum(v for k, v in moved.items() if k != "allgather_densify")
    ufull = sum(alg.values())
    ucore = sum(v for k, v in alg.items() if k != "allgather_densify")
    r = {"bytes": "moved by this design (add stream + candidates, top-k reads of candidates and of fallen-back "
                  "blocks, sparse traffic, decode)",
         "alg_bytes_full": mfull, "achieved_full_GBs": mfull / sec / 1e9, "frac_full": mfull / sec / 1e9 / HBM_PEAK_GBS,
         "alg_bytes_core": mcore, "frac_core": mcore / sec / 1e9 / HBM_PEAK_GBS,
         "unfused_16B_per_element": {"alg_bytes_full": ufull, "frac_full": ufull / sec / 1e9 / HBM_PEAK_GBS,
                                     "alg_bytes_core": ucore, "frac_core": ucore / sec / 1e9 / HBM_PEAK_GBS}}
    if stats is not None:
        r["speculative_candidates"] = cand
        r["blocks_read_again"] = sum(1 for ok in stats["spec_ok"] if not ok)
        r["elements_read_again"] = reread
    return r


# Above this many bytes of residual plus resident gradient batches the
# workload runs one worker at a time (the GPT-2-XL-sized one: 192 GB of residual).
PER_WORKER_BYTES = 200e9
# workers per residual-add / block top-k call there (--rows-per-call): one row
# of workspace (18 GB of candidates) and gradient (6 GB) beside the 192 GB
# residual.  Two rows fit too (selection 1.9 ms faster per step) but the adds
# over the larger footprint lose 2.3 ms.
PER_WORKER_ROWS = 1


def run_per_worker(args, wl, dev) -> int:
    if args.teams > 1:
        print(json.dumps({"error": "the per-worker run (workload 5) has no team variant"}))
        return 2
    R = args.rows_per_call if args.rows_per_call > 0 else PER_WORKER_ROWS
    if wl.P % R:
        print(json.dumps({"error": f"--rows-per-call must divide P = {wl.P}"}))
        return 2
    out = per_worker_measure(wl, dev, args.steps, args.warmup, R, args.variant == "lazy", False)
    print(json.dumps(out), flush=True)
    return 0


def per_worker_measure(wl, dev, steps: int, warmup: int, R: int, lazy: bool, fuse_collect: bool = True) -> dict:
    """A workload whose gradients cannot all be resident beside the residual:
    the workers' gradients are generated on the GPU R at a time (untimed
    input plumbing), then their residual add and block top-k run on a
    workspace for that many rows; the SRS steps, the decode and the residual
    collection follow for all workers.  Step time = the sum of the
    event-timed hot calls (marker cost removed); `span_ms_per_step` is the
    event-timed span of the whole step on the stream, gaps between the calls
    included, less the generation kernels inside it."""
    import torch

    from paper_2304_00737_amd import spardl
    from paper_2304_00737_amd import workloads as W

    P, n, kb = wl.P, wl.n, wl.k_blk
    if lazy:
        st = spardl.SparDLLazyStep(P, n, kb, device=dev, rows_per_call=R)
    else:
        st = spardl.SparDLStep(P, n, kb, device=dev, rows_per_call=R, fuse_collect=fuse_collect)
    gen = W.DeviceGenerator(wl, device=dev)
    g = torch.empty((R, n), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def ev():
        return torch.cuda.Event(enable_timing=True)

    empty = [(ev(), ev()) for _ in range(64)]
    for a, b in empty:
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    marker_ms = sum(a.elapsed_time(b) for a, b in empty) / len(empty)

    def one_step(j, stats=None):
        t = j % wl.steps + 1
        marks, gens = [], []
        s0, s1 = ev(), ev()
        s0.record(stream)
        for w0 in range(0, P, R):
            gg = (ev(), ev())
            gg[0].record(stream)
            for r in range(R):
                gen.fill(g[r], t, w0 + r)
            gg[1].record(stream)
            gens.append(gg)
            e = (ev(), ev(), ev())
            e[0].record(stream)
            st.residual_add_rows(w0, g)
            e[1].record(stream)
            if not lazy:   # the lazy variant selects inside finish(), round by round
                st.block_topk_rows(w0, R)
            e[2].record(stream)
            marks.append(e)
            if stats is not None:   # untimed statistics step: read this worker group's candidates
                stats.append(spardl.topk_stats(st.ws, R, P, n, kb))
        f = (ev(), ev())
        f[0].record(stream)
        st.finish()
        f[1].record(stream)
        s1.record(stream)
        torch.cuda.synchronize()
        ws_check(st)
        add = sum(a.elapsed_time(b) for a, b, _ in marks) - len(marks) * marker_ms
        topk = 0.0 if lazy else sum(b.elapsed_time(c) for _, b, c in marks) - len(marks) * marker_ms
        tail = f[0].elapsed_time(f[1]) - marker_ms
        gen_ms = sum(a.elapsed_time(b) for a, b in gens)
        return add, topk, tail, s0.elapsed_time(s1) - gen_ms

    t0 = time.time()
    for j in range(warmup):
        one_step(j)
    res = [one_step(warmup + j) for j in range(steps)]
    stats = []
    if not lazy:
        one_step(warmup + steps, stats)
    add_ms = sum(r[0] for r in res) / steps
    topk_ms = sum(r[1] for r in res) / steps
    tail_ms = sum(r[2] for r in res) / steps
    span_ms = sum(r[3] for r in res) / steps
    ms_per_step = add_ms + topk_ms + tail_ms
    add_launch_ms = add_ms / (P // R)
    alg_add = 12.0 * R * n
    achieved = alg_add / (add_launch_ms * 1e-3) / 1e9
    # bytes per step: the unfused 16 B per element (read G and xi, write A, read A again for the
    # selection) and what this design moves (the add's 12 B, its candidates, the top-k's reads of
    # them and of blocks it read again, the selections); both with the sparse and decode traffic
    _, _, bags = spardl.srs_plan(P)
    # merges: read held + received, write kept + dropped; decode: write u and the bitmap, read the final
    # blocks; collection: read the local indices and the drops, read and write the entries they touch
    # (upper bound: every drop)
    sparse = 32.0 * P * kb * sum(bags) + (4.0 * n + n / 8.0 + 8.0 * P * kb) + (4.0 * P * P * kb + 16.0 * P * kb * sum(bags))
    unfused = 16.0 * P * n + 12.0 * P * P * kb + sparse
    cand = sum(sum(x["candidates"]) for x in stats)
    blen = [((b + 1) * n) // P - (b * n) // P for b in range(P)]
    reread = sum(blen[u % P] for x in stats for u, ok in enumerate(x["spec_ok"]) if not ok)
    moved = 12.0 * P * n + 16.0 * cand + 4.0 * reread + 12.0 * P * P * kb + sparse
    sec = ms_per_step * 1e-3
    return {
        "metric": (f"gradient elements/sec per full SparDL step, lazy sparsification (P={P} virtual); % of HBM peak"
                   if lazy else f"gradient elements/sec per full SparDL step (P={P} virtual); % of HBM peak"),
        "value": P * n / sec,
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_per_step,
        "span_ms_per_step": span_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "P": P, "n_per_worker": n, "density": f"{wl.density[0]}/{wl.density[1]}",
                   "k_per_block": kb, "gradient_batches": wl.steps, "residual": "carried across steps",
                   "segments": len(wl.seg_len), "seed": W.SEED_BASE, "variant": "lazy" if lazy else "eager",
                   "residual_collection": ("inside the next step's residual add" if getattr(st, "fuse_collect", False)
                                           else "its own call at the end of the step"),
                   "timing": "ms_per_step: sum of the event-timed hot calls; span_ms_per_step: the whole step's "
                             "span on the stream less the gradient generation inside it; the workers' gradients "
                             f"are generated on the GPU between their calls, {R} rows per call ({R}-row workspace)"},
        "roofline": {"bound": "hbm", "kernel": ("k_residual_add4<true, true> (the previous step's collection fused in)"
                                                if getattr(st, "fuse_collect", False) else "k_residual_add4<true, false>"),
                     "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "alg_bytes_per_launch": alg_add, "avg_launch_ms": add_launch_ms},
        "step_roofline": ({"bytes": "moved by this design", "alg_bytes_full": moved,
                           "frac_full": moved / sec / 1e9 / HBM_PEAK_GBS,
                           "speculative_candidates": cand, "elements_read_again": reread,
                           "unfused_16B_per_element": {"alg_bytes_full": unfused,
                                                       "frac_full": unfused / sec / 1e9 / HBM_PEAK_GBS}}
                          if not lazy else
                          {"unfused_16B_per_element": {"alg_bytes_full": unfused,
                                                       "frac_full": unfused / sec / 1e9 / HBM_PEAK_GBS}}),
        "per_call_ms": ({"residual_add_all_workers": add_ms, "rounds_densify_collect": tail_ms} if lazy else
                        {"residual_add_all_workers": add_ms, "block_topk_all_workers": topk_ms,
                         "srs_densify_collect": tail_ms}),
        "event_marker_ms": marker_ms,
        "wall_s": time.time() - t0,
        "kernel_src": _kernel_src_hash(),
    }


def graph_measure(wl, dev, steps: int) -> dict:
    """The launch-bound workload's whole step (about twenty launches of a
    few microseconds each) timed eagerly and replayed from a captured HIP
    graph (the library enqueues kernels only, so the step can be captured;
    tests/test_gpu_graph.py checks replays bit for bit)."""
    import torch

    from paper_2304_00737_amd import spardl
    from paper_2304_00737_amd import workloads as W

    P, n, kb = wl.P, wl.n, wl.k_blk
    gen = W.DeviceGenerator(wl, device=dev)
    g = torch.empty((P, n), dtype=torch.float32, device=dev)
    for w in range(P):
        gen.fill(g[w], 1, w)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    out = {"workload": wl.name, "P": P, "n_per_worker": n, "k_per_block": kb, "steps": steps}
    with torch.cuda.stream(side):
        st = spardl.SparDLStep(P, n, kb, device=dev, fuse_collect=True)
        for _ in range(10):
            st.step(g)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(side)
        for _ in range(steps):
            st.step(g)
        b.record(side)
        torch.cuda.synchronize()
        out["eager_ms_per_step"] = a.elapsed_time(b) / steps
        graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        st.step(g)
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        for _ in range(10):
            graph.replay()
        torch.cuda.synchronize()
        a.record(side)
        for _ in range(steps):
            graph.replay()
        b.record(side)
        torch.cuda.synchronize()
    ws_check(st)
    out["graph_ms_per_step"] = a.elapsed_time(b) / steps
    out["graph_value"] = P * n / (out["graph_ms_per_step"] * 1e-3)
    out["eager_value"] = P * n / (out["eager_ms_per_step"] * 1e-3)
    return out


if __name__ == "__main__":
    sys.exit(main())
