"""Bit-exact block top-k of one worker's row when the call has at least 2^17
candidate slots, the size from which the collect and the emit give each wave
two slots (eight when a block keeps fewer than 8 entries per slot) and the
staged threshold walks 256-slot groups as one list.

One row of 16 blocks of 33,588,228 elements (8201 slots each, the last one
ragged; 16 units of that many slots take the staged threshold), tie-heavy
values (every entry in {+-1, +-2, +-4} x 2^-8, 30 % exact zeros): the
threshold bin holds about a tenth of every block, so the slots are crowded
(their candidate lists run past the preloaded first entries) and the
flattened walks take many rounds.  Two steps of the fused add + block top-k:
the first has no candidates from the add, the second takes them.  The oracle
recomputes sampled blocks."""

import numpy as np
import pytest

from oracle import spardl_oracle as so
from tests.conftest import gpu_available
from tests.gpu_util import assert_bits_equal, assert_idx_equal, log

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    from paper_2304_00737_amd import spardl

P = 16
M = 4096 * 8200 + 1028          # block length: a multiple of 4, not of the 4096-element slot
N = P * M
KB = M // 100
BLOCKS = [0, 15]


def _ties(n, seed):
    rng = np.random.default_rng(seed)
    lut = np.array([1, -1, 2, -2, 4, -4], dtype=np.float32) * np.float32(2.0 ** -8)
    v = lut[rng.integers(0, 6, size=n, dtype=np.uint8)]
    v[rng.random(n, dtype=np.float32) < 0.3] = 0.0
    return v


def _normal(n, seed):
    return np.random.default_rng(seed).standard_normal(n, dtype=np.float32)


@pytest.mark.parametrize("kind,kb", [("ties", KB), ("normal", M // 1000)])
def test_block_topk_many_slots_one_row(kind, kb):
    """ties at 1 %: crowded slots, two slots per wave; N(0,1) at 0.1 %: about
    ten candidates per slot and fewer than 8 kept entries per slot, so eight
    slots per wave."""
    assert P * ((M + 4095) // 4096) >= 1 << 17
    KB = kb
    log(f"many-slot block top-k: one row, P={P}, block {M}, k_blk {KB}, {kind}")
    gen = _ties if kind == "ties" else _normal
    acc = torch.zeros((1, N), dtype=torch.float32, device="cuda")
    ws = spardl.workspace(1, P, N, KB)
    sp_i = torch.empty((1, P, KB), dtype=torch.int32, device="cuda")
    sp_v = torch.empty((1, P, KB), dtype=torch.float32, device="cuda")
    li = torch.empty((1, P, KB), dtype=torch.int32, device="cuda")
    host = np.zeros(N, np.float32)
    for step in range(2):
        g = gen(N, 40 + step)
        spardl.residual_add(acc, torch.from_numpy(g).cuda().view(1, N), 1, N, P, ws, KB)
        spardl.block_topk(acc, 1, N, P, KB, sp_i, sp_v, li, ws, spardl.TOPK_HIST_READY)
        torch.cuda.synchronize()
        assert spardl.ws_error(ws) == 0
        host = host + g   # one fp32 add per element, as on the GPU
        del g
        log(f"  step {step + 1}: GPU done, oracle on blocks {BLOCKS}")
        gi, gv, gl = sp_i[0].cpu().numpy(), sp_v[0].cpu().numpy(), li[0].cpu().numpy()
        for b in BLOCKS:
            oi, ov = so.local_sparsify(host[b * M:(b + 1) * M], b * M, KB)
            assert_idx_equal(gi[b], oi, f"step {step + 1} block {b} idx")
            assert_bits_equal(gv[b], ov, f"step {step + 1} block {b} val")
            assert_idx_equal(gl[b], oi, f"step {step + 1} block {b} local idx")
        log(f"  step {step + 1}: bit-exact")
    del acc, ws, sp_i, sp_v, li
    torch.cuda.empty_cache()
