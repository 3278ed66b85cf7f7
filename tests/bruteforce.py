"""Independent pure-Python brute force of one SparDL step (d = 1), for tiny inputs.

Written separately from the oracle, in a different style (dicts of
index -> fp32 value, Python's sorted(), a closed-form bag layout, and an
explicit per-worker "discarded" ledger for the residual), so that the oracle
can be pinned against it.  It follows the paper (SparDL, arXiv 2304.00737):
Sec. II (top-k), Sec. III-B (partitioning, transmission with sparsification),
Sec. III-C / Algorithm 1 (global residual collection).
"""

from __future__ import annotations

import numpy as np

F32 = np.float32


def _mag(v) -> int:
    return int(np.array([v], dtype=np.float32).view(np.uint32)[0]) & 0x7FFFFFFF


def bf_topk(d: dict, k: int) -> dict:
    """Keep the k entries of largest |v|, ties to the lower index (full sort)."""
    ranked = sorted(d.items(), key=lambda kv: (-_mag(kv[1]), kv[0]))
    return dict(ranked[:k])


def bf_merge(held: dict, recv: dict) -> dict:
    out = dict(held)
    for x, v in recv.items():
        out[x] = F32(out[x] + v) if x in out else F32(v)
    return out


def bf_step(acc_rows, grad_rows, P: int, k: int):
    """Returns (dense u, new residual rows, final dicts per block, drops, local)."""
    n = len(acc_rows[0])
    s = [b * n // P for b in range(P + 1)]
    A = [[F32(F32(acc_rows[w][x]) + F32(grad_rows[w][x])) for x in range(n)] for w in range(P)]

    state = {}
    local = {}
    for w in range(P):
        for b in range(P):
            block = {x: A[w][x] for x in range(s[b], s[b + 1])}
            state[(w, b)] = bf_topk(block, k)
            local[(w, b)] = dict(state[(w, b)])

    l = 0
    while (1 << l) < P:
        l += 1
    drops = {}
    for i in range(1, l + 1):
        dist = 1 << (l - i)
        # bag B_{l-i+1} of worker w sits at circle positions [2^(l-i), 2^(l-i+1)) from w
        lo, hi = 1 << (l - i), min(1 << (l - i + 1), P)
        inbox = {}
        for w in range(P):
            dst = (w + dist) % P
            inbox[dst] = [(b, dict(state[(w, b)])) for b in ((w + t) % P for t in range(lo, hi))]
        for r in range(P):
            for b, msg in inbox[r]:
                merged = bf_merge(state[(r, b)], msg)
                kept = bf_topk(merged, k)
                state[(r, b)] = kept
                drops[(i, r, b)] = {x: v for x, v in merged.items() if x not in kept}

    final = {b: state[(b, b)] for b in range(P)}
    u = [F32(0.0)] * n
    for b in range(P):
        for x, v in final[b].items():
            u[x] = v
    I = set()
    for b in range(P):
        I |= set(final[b].keys())

    new_res = []
    for w in range(P):
        ledger = {}
        for x in range(n):
            b = next(bb for bb in range(P) if s[bb] <= x < s[bb + 1])
            if x not in local[(w, b)]:
                ledger[x] = A[w][x]
        for i in range(1, l + 1):
            for (ii, ww, b), d in drops.items():
                if ii == i and ww == w:
                    for x, v in d.items():
                        ledger[x] = F32(ledger.get(x, F32(0.0)) + v)
        row = []
        for x in range(n):
            row.append(ledger.get(x, F32(0.0)) if x in I else A[w][x])
        new_res.append(row)
    return u, new_res, final, drops, local


def bf_step_lazy(acc_rows, grad_rows, P: int, k: int):
    """Lazy sparsification (Sec. III-B "Optimization for SRS", Algorithm 1):
    dense per-worker rows, each block sparsified once, right before it is sent
    (or at the end for the reserved block).

    Returns (dense u, new residual rows, final dicts per block, selections
    {(w, b): dict}).  The residual is built from a per-worker record of what
    the worker still held (unsent) at each index when it gave the block up.
    """
    n = len(acc_rows[0])
    s = [b * n // P for b in range(P + 1)]
    A = [[F32(F32(acc_rows[w][x]) + F32(grad_rows[w][x])) for x in range(n)] for w in range(P)]
    cur = [list(row) for row in A]          # the dense blocks each worker works on
    l = 0
    while (1 << l) < P:
        l += 1
    sel = {}
    left_behind = [dict() for _ in range(P)]   # x -> value w kept back when it sparsified x's block

    def sparsify(w, b):
        block = {x: cur[w][x] for x in range(s[b], s[b + 1])}
        kept = bf_topk(block, k)
        sel[(w, b)] = kept
        for x, v in block.items():
            left_behind[w][x] = F32(0.0) if x in kept else v
        return kept

    for i in range(1, l + 1):
        dist = 1 << (l - i)
        lo, hi = 1 << (l - i), min(1 << (l - i + 1), P)
        inbox = {}
        for w in range(P):
            inbox[(w + dist) % P] = [(b, dict(sparsify(w, b))) for b in ((w + t) % P for t in range(lo, hi))]
        for r in range(P):
            for b, msg in inbox[r]:
                for x, v in msg.items():
                    cur[r][x] = F32(cur[r][x] + v)
    for w in range(P):
        sparsify(w, w)

    final = {b: sel[(b, b)] for b in range(P)}
    u = [F32(0.0)] * n
    I = set()
    for b in range(P):
        for x, v in final[b].items():
            u[x] = v
            I.add(x)
    new_res = [[left_behind[w][x] if x in I else A[w][x] for x in range(n)] for w in range(P)]
    return u, new_res, final, sel


def bf_step_rsag(acc_rows, grad_rows, P: int, L: int, d: int):
    """d teams of Q = P / d consecutive workers: SRS inside each team over Q
    blocks, then recursive doubling across teams (partner team X xor 2^t) with
    top-L after each exchange; every worker records the drops of its merge and
    takes 1 / (workers that made the same merge) = 2^-(t+1) of each into its
    residual (Sec. III-D).

    Returns (dense u, new residual rows, final dicts per block).
    """
    n = len(acc_rows[0])
    Q = P // d
    s = [b * n // Q for b in range(Q + 1)]
    A = [[F32(F32(acc_rows[w][x]) + F32(grad_rows[w][x])) for x in range(n)] for w in range(P)]
    state, local, ledger_drops = {}, {}, [dict() for _ in range(P)]   # x -> list of drop values, in order
    for w in range(P):
        for b in range(Q):
            state[(w, b)] = bf_topk({x: A[w][x] for x in range(s[b], s[b + 1])}, L)
            local[(w, b)] = dict(state[(w, b)])
    l = 0
    while (1 << l) < Q:
        l += 1
    for i in range(1, l + 1):
        dist = 1 << (l - i)
        lo, hi = 1 << (l - i), min(1 << (l - i + 1), Q)
        for tau in range(d):
            inbox = {}
            for q in range(Q):
                dst = (q + dist) % Q
                inbox[dst] = [(b, dict(state[(tau * Q + q, b)])) for b in ((q + t) % Q for t in range(lo, hi))]
            for r in range(Q):
                w = tau * Q + r
                for b, msg in inbox[r]:
                    merged = bf_merge(state[(w, b)], msg)
                    kept = bf_topk(merged, L)
                    state[(w, b)] = kept
                    for x, v in merged.items():
                        if x not in kept:
                            ledger_drops[w].setdefault(x, []).append(v)
    t = 0
    while (1 << t) < d:
        new = {}
        for w in range(P):
            X, q = divmod(w, Q)
            partner = (X ^ (1 << t)) * Q + q
            merged = bf_merge(state[(w, q)], state[(partner, q)])
            new[w] = (bf_topk(merged, L), merged)
        for w in range(P):
            kept, merged = new[w]
            state[(w, w % Q)] = kept
            for x, v in merged.items():
                if x not in kept:
                    ledger_drops[w].setdefault(x, []).append(F32(v * F32(1.0 / (2 << t))))
        t += 1
    final = {b: state[(b, b)] for b in range(Q)}
    for w in range(P):
        assert state[(w, w % Q)] == final[w % Q]
    u = [F32(0.0)] * n
    I = set()
    for b in range(Q):
        for x, v in final[b].items():
            u[x] = v
            I.add(x)
    new_res = []
    for w in range(P):
        row = []
        for x in range(n):
            if x not in I:
                row.append(A[w][x])
                continue
            b = next(bb for bb in range(Q) if s[bb] <= x < s[bb + 1])
            r = F32(0.0) if x in local[(w, b)] else A[w][x]
            for v in ledger_drops[w].get(x, []):
                r = F32(r + v)
            row.append(r)
        new_res.append(row)
    return u, new_res, final


class BfController:
    """Algorithm 2 restated: returns the top-h count for the next step."""

    def __init__(self, L, d):
        self.L, self.d = L, d
        self.state = {"h": L / d, "step": 0.01 * (d - 1) * L / d, "flag": False, "N": 0}

    def count(self):
        s = self.state
        too_many = s["N"] > self.L
        rising = s["step"] > 0
        if too_many == rising:          # the xor is false: turn round, halve
            s["step"] = -s["step"] * 0.5
            s["flag"] = False
        elif s["flag"]:                 # second step the same way in a row: double
            s["step"] = s["step"] * 2.0
            s["flag"] = False
        else:
            s["flag"] = True
        s["h"] = min(max(s["h"] + s["step"], self.L / self.d), float(self.L))
        c = int(s["h"] + 0.5)
        return min(max(c, 1), self.L)


def bf_step_bsag(acc_rows, grad_rows, P: int, L: int, d: int, ctrls: dict):
    """d teams of Q = P / d consecutive workers: SRS inside each team, top-h of
    each held block, all-gather across teams summed in team order, top-L when
    more than L indices result (Sec. III-D, Algorithm 2 for h).

    Returns (dense u, new residual rows, final dicts per block, counts h per
    block, union sizes per block).
    """
    n = len(acc_rows[0])
    Q = P // d
    s = [b * n // Q for b in range(Q + 1)]
    A = [[F32(F32(acc_rows[w][x]) + F32(grad_rows[w][x])) for x in range(n)] for w in range(P)]
    state, local, ledger = {}, {}, [dict() for _ in range(P)]
    for w in range(P):
        for b in range(Q):
            state[(w, b)] = bf_topk({x: A[w][x] for x in range(s[b], s[b + 1])}, L)
            local[(w, b)] = dict(state[(w, b)])
    l = 0
    while (1 << l) < Q:
        l += 1
    for i in range(1, l + 1):
        dist = 1 << (l - i)
        lo, hi = 1 << (l - i), min(1 << (l - i + 1), Q)
        for tau in range(d):
            inbox = {}
            for q in range(Q):
                inbox[(q + dist) % Q] = [(b, dict(state[(tau * Q + q, b)])) for b in ((q + t) % Q for t in range(lo, hi))]
            for r in range(Q):
                w = tau * Q + r
                for b, msg in inbox[r]:
                    merged = bf_merge(state[(w, b)], msg)
                    kept = bf_topk(merged, L)
                    state[(w, b)] = kept
                    for x, v in merged.items():
                        if x not in kept:
                            ledger[w].setdefault(x, []).append(v)
    final, hs, Ns = {}, {}, {}
    for q in range(Q):
        c = ctrls.setdefault(q, BfController(L, d)).count()
        hs[q] = c
        gathered = []
        for tau in range(d):
            w = tau * Q + q
            top = bf_topk(state[(w, q)], c)
            for x, v in state[(w, q)].items():
                if x not in top:
                    ledger[w].setdefault(x, []).append(v)
            gathered.append(top)
        total = dict(gathered[0])
        for g in gathered[1:]:
            total = bf_merge(total, g)
        Ns[q] = len(total)
        ctrls[q].state["N"] = len(total)
        final[q] = bf_topk(total, L)
    u = [F32(0.0)] * n
    I = set()
    for q in range(Q):
        for x, v in final[q].items():
            u[x] = v
            I.add(x)
    new_res = []
    for w in range(P):
        row = []
        for x in range(n):
            if x not in I:
                row.append(A[w][x])
                continue
            b = next(bb for bb in range(Q) if s[bb] <= x < s[bb + 1])
            r = F32(0.0) if x in local[(w, b)] else A[w][x]
            for v in ledger[w].get(x, []):
                r = F32(r + v)
            row.append(r)
        new_res.append(row)
    return u, new_res, final, hs, Ns
