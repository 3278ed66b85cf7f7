"""The whole step captured in a HIP graph.  The library enqueues kernels only
(no memset or copy nodes, no host synchronisation), so a captured step must
replay correctly: each replay gets new gradients copied into the captured
input buffer, with eager work and a synchronisation between replays, and must
match an eager twin bit for bit every time (the residual, and for B-SAG the
controller of Algorithm 2, carry over from replay to replay)."""

import numpy as np
import pytest

from tests.conftest import gpu_available
from tests.gpu_util import assert_bits_equal, assert_idx_equal, log

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    from paper_2304_00737_amd import spardl
    from paper_2304_00737_amd import workloads as W

CASES = {
    "eager": (4, 1 << 18, 300),
    "lazy": (4, 1 << 18, 300),
    "rsag": (8, 1 << 18, 600),
    "bsag": (6, 200003, 450),
}


def _make(kind, P, n, kb):
    if kind == "eager":
        return spardl.SparDLStep(P, n, kb)
    if kind == "lazy":
        return spardl.SparDLLazyStep(P, n, kb)
    if kind == "rsag":
        return spardl.SparDLSagStep(P, 2, n, kb)
    return spardl.SparDLSagStep(P, 3, n, kb, bruck=True)


def _errors(st):
    ws = [getattr(st, a) for a in ("ws", "ws_sag") if hasattr(st, a)] + list(getattr(st, "ws_team", []))
    return [spardl.ws_error(w) for w in ws]


@pytest.mark.parametrize("kind", list(CASES))
def test_captured_step_replays(kind):
    P, n, kb = CASES[kind]
    log(f"graph capture of the {kind} step P={P} n={n} kb={kb}")
    g_st, e_st = _make(kind, P, n, kb), _make(kind, P, n, kb)
    gbuf = torch.empty((P, n), dtype=torch.float32, device="cuda")
    grads = [torch.from_numpy(W.small_rows("normal", P, n, 900 + t)).cuda() for t in range(6)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # one eager step on both before the capture
        gbuf.copy_(grads[0])
        g_st.step(gbuf)
        e_st.step(grads[0])
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        g_st.step(gbuf)
    torch.cuda.synchronize()
    for t in range(1, 6):
        gbuf.copy_(grads[t])
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        e_st.step(grads[t])
        torch.cuda.synchronize()
        assert _errors(g_st) == [0] * len(_errors(g_st)) and not any(_errors(e_st))
        assert_bits_equal(g_st.dense.cpu().numpy(), e_st.dense.cpu().numpy(), f"replay {t}: dense")
        assert_bits_equal(g_st.acc.cpu().numpy().ravel(), e_st.acc.cpu().numpy().ravel(), f"replay {t}: residual")
        assert_idx_equal(g_st.sp_idx.cpu().numpy(), e_st.sp_idx.cpu().numpy(), f"replay {t}: sparse indices")
        assert_bits_equal(g_st.sp_val.cpu().numpy().ravel(), e_st.sp_val.cpu().numpy().ravel(),
                          f"replay {t}: sparse values")
        _ = torch.ones(4096, device="cuda").sum().item()   # eager work between replays
    log("  5 replays bit-exact")
