"""Throughput of one full SparDL synchronisation step (d = 1) on one MI355X.

A step is the whole hot path for P simulated workers over one batch of
gradients: residual add (fused level-1 histogram), block top-k/P, the
ceil(log2 P) Spar-Reduce-Scatter steps, the All-Gather decode to a dense
update, and global residual collection.  The default workload is the
ResNet-50-sized one: P = 8, n = 25.6M fp32 per worker, density 1%, three
distinct gradient batches cycled with the residual carried across steps.
Inputs are generated on the host and resident in HBM before timing starts.

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


def cpu_baseline(wl, max_seconds: float = 25.0, lazy: bool = False):
    """The oracle, as it stands, on a bounded sample of the same workload:
    whole block indices (blocks never interact, so a block index is a
    self-contained unit of a step), each through the workload's steps with its
    residual carried, until about max_seconds of oracle time."""
    import numpy as np

    from oracle import spardl_oracle as so
    from paper_2304_00737_amd import workloads as W

    P, n, kb = wl.P, wl.n, wl.k_blk
    bounds = so.block_bounds(n, P)
    done_elems, elapsed, units = 0, 0.0, 0
    step_fn = so.spardl_step_lazy if lazy else so.spardl_step
    for b in range(P):
        acc = [{b: np.zeros(bounds[b + 1] - bounds[b], np.float32)} for _ in range(P)]
        for t in range(1, wl.steps + 1):
            grad = [{b: W.gradient(wl, t, w, bounds[b], bounds[b + 1] - bounds[b])} for w in range(P)]
            t0 = time.perf_counter()
            step_fn(acc, grad, P, n, kb, blocks=[b])
            elapsed += time.perf_counter() - t0
            done_elems += P * (bounds[b + 1] - bounds[b])
            units += 1
            if elapsed > max_seconds:
                break
        if elapsed > max_seconds:
            break
    return {"value": done_elems / elapsed, "unit": "elements/s", "cores": 1, "kind": "oracle",
            "sample": f"{units} (block index, step) units of the same workload's {P} block indices x "
                      f"{wl.steps} steps, block by block with the residual carried ({done_elems} gradient "
                      f"elements, {elapsed:.1f} s; numpy, single thread)"}


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
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true",
                    help="first run one untimed device-to-device copy of CALIB_BYTES (a reference "
                         "kernel of known traffic for hardware-counter runs)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs the P simulated workers on one GPU; "
                                   "--gpus must be 1 (no multi-GPU path is built)"}))
        return 2

    import numpy as np
    import torch

    from paper_2304_00737_amd import spardl
    from paper_2304_00737_amd import workloads as W

    wl = W.config(args.workload)
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
        st = spardl.SparDLStep(P, n, kb, device=dev)
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

    # ---- dominant kernel: the residual add is one kernel per call; each
    # launch is bracketed by an event pair on its stream (marker cost removed)
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
    torch.cuda.synchronize()
    add_ms = sum(a.elapsed_time(b) for a, b in k_mid) / args.steps - marker_ms
    ws_check(st)

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
                   "L_per_team_block": st.k_blk if d > 1 else None},
        "roofline": {"bound": "hbm", "kernel": "k_residual_add" if dominant == "residual_add" else dominant,
                     "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "alg_bytes_per_launch": alg[dominant], "avg_launch_ms": dom_ms},
        "step_roofline": {"alg_bytes_full": full_bytes, "alg_bytes_core": core_bytes,
                          "achieved_full_GBs": full_bytes / (ms_per_step * 1e-3) / 1e9,
                          "frac_full": full_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS},
        "per_call_ms": per_call_ms,
        "event_marker_ms": marker_ms,
        "wall_s_timed": wall,
        "kernel_src": src_hash,
    }
    if not args.no_cpu_baseline and d == 1:
        out["cpu_baseline"] = cpu_baseline(wl, lazy=lazy)
    print(json.dumps(out), flush=True)
    return 0


# Above this many bytes of residual plus resident gradient batches the
# workload runs one worker at a time (the GPT-2-XL-sized one: 192 GB of residual).
PER_WORKER_BYTES = 200e9
# workers per residual-add / block top-k call there (--rows-per-call): one row
# of workspace (18 GB of candidates) and gradient (6 GB) beside the 192 GB
# residual.  Two rows fit too (selection 1.9 ms faster per step) but the adds
# over the larger footprint lose 2.3 ms.
PER_WORKER_ROWS = 1


def run_per_worker(args, wl, dev) -> int:
    """A workload whose gradients cannot all be resident beside the residual:
    the workers' gradients are generated on the GPU PER_WORKER_ROWS at a time
    (untimed), then their residual add and block top-k run on a workspace for
    that many rows; the SRS steps, the decode and the residual collection
    follow for all workers.  Step time = the sum of the event-timed hot calls
    (marker cost removed)."""
    import torch

    from paper_2304_00737_amd import spardl
    from paper_2304_00737_amd import workloads as W

    P, n, kb = wl.P, wl.n, wl.k_blk
    if args.teams > 1:
        print(json.dumps({"error": "the per-worker run (workload 5) has no team variant"}))
        return 2
    lazy = args.variant == "lazy"
    R = args.rows_per_call if args.rows_per_call > 0 else PER_WORKER_ROWS
    if P % R:
        print(json.dumps({"error": f"--rows-per-call must divide P = {P}"}))
        return 2
    if lazy:
        st = spardl.SparDLLazyStep(P, n, kb, device=dev, rows_per_call=R)
    else:
        st = spardl.SparDLStep(P, n, kb, device=dev, rows_per_call=R)
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

    def one_step(j):
        t = j % wl.steps + 1
        marks = []
        for w0 in range(0, P, R):
            for r in range(R):
                gen.fill(g[r], t, w0 + r)
            e = (ev(), ev(), ev())
            e[0].record(stream)
            st.residual_add_rows(w0, g)
            e[1].record(stream)
            if not lazy:   # the lazy variant selects inside finish(), round by round
                st.block_topk_rows(w0, R)
            e[2].record(stream)
            marks.append(e)
        f = (ev(), ev())
        f[0].record(stream)
        st.finish()
        f[1].record(stream)
        torch.cuda.synchronize()
        ws_check(st)
        add = sum(a.elapsed_time(b) for a, b, _ in marks) - len(marks) * marker_ms
        topk = 0.0 if lazy else sum(b.elapsed_time(c) for _, b, c in marks) - len(marks) * marker_ms
        tail = f[0].elapsed_time(f[1]) - marker_ms
        return add, topk, tail

    warm = max(1, min(args.warmup, 2))
    steps = max(1, min(args.steps, 3))
    t0 = time.time()
    for j in range(warm):
        one_step(j)
    res = [one_step(warm + j) for j in range(steps)]
    add_ms = sum(r[0] for r in res) / steps
    topk_ms = sum(r[1] for r in res) / steps
    tail_ms = sum(r[2] for r in res) / steps
    ms_per_step = add_ms + topk_ms + tail_ms
    add_launch_ms = add_ms / (P // R)
    alg_add = 12.0 * R * n
    achieved = alg_add / (add_launch_ms * 1e-3) / 1e9
    full = 16.0 * P * n + 4.0 * n + n / 8.0 + 12.0 * P * P * kb
    out = {
        "metric": ("gradient elements/sec per full SparDL step, lazy sparsification (P=8 virtual); % of HBM peak"
                   if lazy else "gradient elements/sec per full SparDL step (P=8 virtual); % of HBM peak"),
        "value": P * n / (ms_per_step * 1e-3),
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warm,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "P": P, "n_per_worker": n, "density": f"{wl.density[0]}/{wl.density[1]}",
                   "k_per_block": kb, "gradient_batches": wl.steps, "residual": "carried across steps",
                   "segments": len(wl.seg_len), "seed": W.SEED_BASE, "variant": args.variant,
                   "timing": "sum of event-timed hot calls; the workers' gradients generated on the GPU "
                             f"between them, {R} rows per call ({R}-row workspace)"},
        "roofline": {"bound": "hbm", "kernel": "k_residual_add", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "alg_bytes_per_launch": alg_add, "avg_launch_ms": add_launch_ms},
        "step_roofline": {"alg_bytes_full": full, "achieved_full_GBs": full / (ms_per_step * 1e-3) / 1e9,
                          "frac_full": full / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS},
        "per_call_ms": ({"residual_add_all_workers": add_ms, "rounds_densify_collect": tail_ms} if lazy else
                        {"residual_add_all_workers": add_ms, "block_topk_all_workers": topk_ms,
                         "srs_densify_collect": tail_ms}),
        "event_marker_ms": marker_ms,
        "wall_s": time.time() - t0,
        "kernel_src": _kernel_src_hash(),
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
