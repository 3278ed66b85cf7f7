"""Non-finite and extreme values through every step of the hot path (block
top-k, the SRS merges, the decode and the residual collection), compared with
the oracle over several steps with the residual carried.

Selection ranks |v| as the bit pattern with the sign cleared, so +Inf ranks
above every finite value, NaNs above +Inf, and -0 equals +0 (ties then go to
the lower index); subnormals are kept (no flush to zero).

Infinities, merge sums that overflow to infinity, signed zeros and
subnormals are compared bit for bit.  A NaN that arithmetic creates
(Inf + -Inf in a merge) or propagates has a sign and payload IEEE 754 leaves
to the implementation, and x86 and gfx950 differ there, so the NaN cases
compare indices exactly and values as "both NaN" where the oracle has a NaN
(every other value bit for bit); fewer NaNs than k/P per block keep the
selected sets independent of the order among NaNs.
"""

import numpy as np
import pytest

import tests.gpu_util as gu
from oracle import spardl_oracle as so
from tests.conftest import gpu_available
from tests.gpu_util import check_ws, compare_step, log

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    from paper_2304_00737_amd import spardl

F32 = np.float32


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _inf_rows(P, n, seed):
    """Normal rows with +-Inf (some at an index shared by every worker, same
    sign), +-3e38 at shared indices (the merges overflow to +-Inf) and one
    block of signed zeros and subnormals whose threshold falls in their ties."""
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((P, n)).astype(F32)
    bounds = so.block_bounds(n, P)
    for w in range(P):
        v[w, rng.choice(n, 6, replace=False)] = F32(np.inf)
        v[w, rng.choice(n, 6, replace=False)] = F32(-np.inf)
    shared = rng.choice(n, 12, replace=False)
    v[:, shared[:3]] = F32(np.inf)
    v[:, shared[3:6]] = F32(-np.inf)
    v[:, shared[6:9]] = F32(3e38)
    v[:, shared[9:]] = F32(-3e38)
    # block 1: signed zeros and subnormals, a few of them drawn per entry
    lo, hi = bounds[1], bounds[2]
    tiny = np.array([0.0, -0.0, 1e-45, -1e-45, 2e-45, -2e-45, 1e-40, -1e-40], F32)
    v[:, lo:hi] = tiny[rng.integers(0, len(tiny), (P, hi - lo))]
    return v


def _nan_rows(P, n, seed):
    """Normal rows with a few quiet NaNs (several payloads, both signs) per
    worker, and +Inf on worker 0 / -Inf on worker 1 at shared indices, so
    that a merge adds Inf and -Inf."""
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((P, n)).astype(F32)
    nan_bits = np.array([0x7FC00000, 0xFFC00000, 0x7FC00001, 0x7FD00000], np.uint32)
    for w in range(P):
        pos = rng.choice(n, 4, replace=False)
        v[w, pos] = nan_bits[rng.integers(0, len(nan_bits), 4)].view(F32)
    shared = rng.choice(n, 4, replace=False)
    v[0, shared] = F32(np.inf)
    v[1, shared] = F32(-np.inf)
    return v


def _nan_aware_bits_equal(got, want, what):
    g = np.ascontiguousarray(np.asarray(got, dtype=F32))
    w = np.ascontiguousarray(np.asarray(want, dtype=F32))
    assert g.shape == w.shape, f"{what}: shapes {g.shape} vs {w.shape}"
    wn = np.isnan(w)
    assert np.array_equal(np.isnan(g), wn), f"{what}: NaN positions differ"
    assert np.array_equal(g.view(np.uint32)[~wn], w.view(np.uint32)[~wn]), f"{what}: values differ"


def _final_residual(st, acc, eq) -> None:
    """With the collection left to the next add: run it, then compare acc."""
    st.flush()
    check_ws(st)
    for w in range(st.P):
        eq(st.acc[w].cpu().numpy(), acc[w], f"residual after flush worker {w}")


# fc: each step's residual collection inside the next step's add (the residual is compared after a flush)
@pytest.mark.parametrize("fc", [False, True])
@pytest.mark.parametrize("P,n,kb", [(4, 40000, 60), (5, 30011, 25)])
def test_infinities_overflow_zeros_subnormals_bit_exact(P, n, kb, fc):
    log(f"non-finite step P={P} n={n} kb={kb} fused collection={fc}: +-Inf, overflowing merges, signed zeros, "
        f"subnormals")
    st = spardl.SparDLStep(P, n, kb, fuse_collect=fc)
    acc = np.zeros((P, n), F32)
    with np.errstate(over="ignore", invalid="ignore"):
        for t in range(3):
            grad = _inf_rows(P, n, 40 + 7 * t + P)
            st.step(_dev(grad))
            check_ws(st)
            res = so.spardl_step([acc[w] for w in range(P)], [grad[w] for w in range(P)], P, n, kb)
            compare_step(st, res, P, n, kb, residual=not fc)
            dense = st.dense.cpu().numpy()
            assert np.isinf(dense).any(), "infinities reach the update"
    if fc:
        _final_residual(st, acc, gu.assert_bits_equal)


@pytest.mark.parametrize("fc", [False, True])
@pytest.mark.parametrize("P,n,kb", [(4, 40000, 60), (3, 20011, 30)])
def test_nans_positions_exact(P, n, kb, fc, monkeypatch):
    log(f"NaN step P={P} n={n} kb={kb} fused collection={fc}: NaN inputs and Inf + -Inf in a merge")
    monkeypatch.setattr(gu, "assert_bits_equal", _nan_aware_bits_equal)
    st = spardl.SparDLStep(P, n, kb, fuse_collect=fc)
    acc = np.zeros((P, n), F32)
    with np.errstate(over="ignore", invalid="ignore"):
        for t in range(2):
            grad = _nan_rows(P, n, 90 + 5 * t + P)
            st.step(_dev(grad))
            check_ws(st)
            res = so.spardl_step([acc[w] for w in range(P)], [grad[w] for w in range(P)], P, n, kb)
            compare_step(st, res, P, n, kb, residual=not fc)
            assert np.isnan(st.dense.cpu().numpy()).any(), "NaNs reach the update"
    if fc:
        _final_residual(st, acc, _nan_aware_bits_equal)
