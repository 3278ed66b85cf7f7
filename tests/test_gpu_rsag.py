"""Bit-exact parity of SparDL with d teams joined by R-SAG (Sec. III-D, d a
power of 2) through the C ABI with the CPU oracle's spardl_step_rsag: the
teams' SRS state and drops, every exchange's drops, the dense update, the
bitmap of the final indices and the residuals, over consecutive steps."""

import numpy as np
import pytest

from oracle import spardl_oracle as so
from tests.conftest import gpu_available
from tests.gpu_util import check_ws, compare_sag_step, log

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    from paper_2304_00737_amd import spardl
    from paper_2304_00737_amd import workloads as W


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _check_sag_ws(st):
    assert spardl.ws_error(st.ws_sag) == 0
    for ws in st.ws_team:
        assert spardl.ws_error(ws) == 0


CASES = [
    # P, d, n, L, kind, steps, fused
    (2, 2, 5000, 40, "normal", 2, True),
    (4, 2, 8192, 100, "ties", 2, True),
    (4, 4, 3001, 7, "dyadic", 2, True),
    (8, 2, 40000, 250, "normal", 3, True),
    (8, 4, 20011, 1, "ties", 2, False),
    (8, 8, 9000, 60, "dyadic", 2, True),
    (12, 4, 30000, 333, "normal", 2, True),
    (16, 8, 16384, 2048, "dyadic", 1, True),   # L = block length: an exact all-reduce
    (16, 16, 5000, 9, "const", 2, True),
    (6, 2, 10007, 3, "zeros", 1, False),
]


@pytest.mark.parametrize("P,d,n,L,kind,steps,fused,batched",
                         [c + (True,) for c in CASES] + [CASES[i] + (False,) for i in (3, 4, 6)])
def test_rsag_step(P, d, n, L, kind, steps, fused, batched):
    """batched: the teams' add, top-k and SRS steps over all P rows in one
    call each; otherwise team by team."""
    log(f"rsag step P={P} d={d} n={n} L={L} kind={kind} steps={steps} fused={fused} batched={batched}")
    st = spardl.SparDLSagStep(P, d, n, L, fused=fused, batched=batched)
    acc = np.zeros((P, n), np.float32)
    for t in range(steps):
        grad = W.small_rows(kind, P, n, 100 * t + 13 * P + d)
        st.step(_dev(grad))
        torch.cuda.synchronize()
        _check_sag_ws(st)
        res = so.spardl_step_rsag([acc[w] for w in range(P)], [grad[w] for w in range(P)], P, n, L, d)
        compare_sag_step(st, res)


@pytest.mark.parametrize("d", [2, 4, 8])
def test_rsag_resnet50_sized(d):
    """The ResNet-50-sized workload (P = 8, n = 25.6M, 1 %) with d teams,
    L = d k / P; the oracle recomputes two block indices of every output."""
    wl = W.config(2)
    P, n = wl.P, wl.n
    Q = P // d
    k = wl.k_blk * P
    L = d * k // P
    log(f"rsag {wl.describe()} d={d} L={L}")
    blocks = [0, Q - 1] if Q > 1 else [0]
    bounds = so.block_bounds(n, Q)
    st = spardl.SparDLSagStep(P, d, n, L)
    grad_d = torch.empty((P, n), dtype=torch.float32, device="cuda")
    host = torch.empty(n, dtype=torch.float32).pin_memory()
    acc = [{b: np.zeros(bounds[b + 1] - bounds[b], np.float32) for b in blocks} for _ in range(P)]
    for t in range(1, 3):
        grad = [dict() for _ in range(P)]
        for w in range(P):
            W.fill(host.numpy(), wl, t, w)
            grad_d[w].copy_(host)
            torch.cuda.synchronize()
            for b in blocks:
                grad[w][b] = host.numpy()[bounds[b]:bounds[b + 1]].copy()
        st.step(grad_d)
        torch.cuda.synchronize()
        _check_sag_ws(st)
        log(f"  step {t}: GPU done, oracle on block indices {blocks}")
        res = so.spardl_step_rsag(acc, grad, P, n, L, d, blocks=blocks)
        compare_sag_step(st, res, blocks=blocks)
        log(f"  step {t}: bit-exact")
