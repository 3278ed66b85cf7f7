"""Bit-exact parity on every block index of the full-size workloads, in the
launch configuration the benchmark uses, against checksums the oracle
produced on the CPU (tests/golden/full_digests.py; tests/digest.py defines
the output streams and the checksum).

Covered: the VGG-16-, BERT- and GPT-2-XL-sized workloads (eager and lazy
sparsification; eager also with each step's residual collection left to the
next step's add, compared with the same checksums: every output of every
step but the pending residual, and the residual after the last step's
flush) and the ResNet-50-sized workload with d = 2, 4, 8 teams joined by
R-SAG and by B-SAG, every step of each with the residual carried.
Besides the checksums, the membership bitmap of the final index set is
compared with the final blocks the GPU holds, and B-SAG's final blocks with
their sentinel padding, on the device.
"""

import json
import os

import numpy as np
import pytest

from oracle import spardl_oracle as so
from tests.conftest import gpu_available
from tests.gpu_util import check_ws, log

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    from paper_2304_00737_amd import spardl
    from paper_2304_00737_amd import workloads as W
    from tests.digest import device_digest, device_streams

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
CASES = [(3, "eager", 1), (4, "eager", 1), (5, "eager", 1), (3, "eager_fc", 1), (4, "eager_fc", 1), (5, "eager_fc", 1),
         (3, "lazy", 1), (4, "lazy", 1), (5, "lazy", 1),
         (2, "rsag", 2), (2, "rsag", 4), (2, "rsag", 8), (2, "bsag", 2), (2, "bsag", 4), (2, "bsag", 8)]
INT32_MAX = 2 ** 31 - 1


def _gold(workload, form, d):
    suffix = f"_d{d}" if form in ("rsag", "bsag") else ""
    path = os.path.join(GOLDEN, f"digests_w{workload}_{form}{suffix}.json")
    if not os.path.exists(path):
        pytest.skip(f"{os.path.basename(path)} not generated")
    return json.load(open(path))


def _check_member(st, finals, n):
    """The bitmap the decode wrote equals the one of the final blocks' indices."""
    idx = torch.cat([f.reshape(-1) for f in finals]).to(torch.int64)
    want = torch.zeros((n + 31) // 32, dtype=torch.int64, device=idx.device)
    want.index_put_((idx >> 5,), torch.ones_like(idx) << (idx & 31), accumulate=True)   # distinct indices: sum = or
    got = st.member.to(torch.int64) & 0xFFFFFFFF
    assert torch.equal(got, want), "membership bitmap differs from the final blocks"


def _run(workload, form, d):
    fc = form == "eager_fc"   # the same outputs as the eager form
    form = "eager" if fc else form
    gold = _gold(workload, form, d)
    wl = W.config(workload)
    P, n, kb = wl.P, wl.n, wl.k_blk
    nb = P if d == 1 else P // d
    assert gold["P"] == P and gold["n"] == n and gold["teams"] == d and gold["blocks_per_row"] == nb
    done = sorted(int(b) for b in gold["digests"])   # a file still being written holds some of them
    assert done and set(done) <= set(range(nb)), done
    bounds = so.block_bounds(n, nb)
    assert gold["bounds"] == [int(x) for x in bounds]
    log(f"full digests: {wl.describe()} form={form} d={d}: {len(done)} of {nb} block indices")
    torch.cuda.empty_cache()
    gen = W.DeviceGenerator(wl)
    per_worker = 4.0 * P * n * 2 > 100e9   # the GPT-2-XL-sized rows: one worker's gradient at a time, as bench.py
    if form in ("rsag", "bsag"):
        st = spardl.SparDLSagStep(P, d, n, d * kb, bruck=form == "bsag")
    elif form == "lazy":
        st = spardl.SparDLLazyStep(P, n, kb, rows_per_call=1 if per_worker else 0)
    else:
        st = spardl.SparDLStep(P, n, kb, rows_per_call=1 if per_worker else 0, fuse_collect=fc)
    g = torch.empty((1 if per_worker else P, n), dtype=torch.float32, device="cuda")
    for t in range(1, wl.steps + 1):
        if per_worker:
            for w in range(P):
                gen.fill(g[0], t, w)
                st.residual_add_rows(w, g)
                if form == "eager":
                    st.block_topk_rows(w, 1)
            st.finish()
        else:
            for w in range(P):
                gen.fill(g[w], t, w)
            st.step(g)
        pending = fc and t < wl.steps   # the residual is collected by the next step's add
        if fc and not pending:
            st.flush()
        torch.cuda.synchronize()
        if form in ("rsag", "bsag"):
            for ws in st.ws_team + [st.ws_sag]:
                assert spardl.ws_error(ws) == 0, "workspace error word"
        else:
            check_ws(st)
        bad = []
        for b in done:
            lo, hi = int(bounds[b]), int(bounds[b + 1])
            streams = device_streams(form, st, P, b, lo, hi, Q=nb, d=d)
            if pending:
                del streams["residual"]
            got = device_digest(streams)
            want = dict(gold["digests"][str(b)][t - 1])
            if pending:
                del want["residual"]
            assert set(got) == set(want), (sorted(got), sorted(want))
            bad += [(b, k) for k in want if got[k] != want[k]]
        assert not bad, f"step {t}: (block index, output) checksums differ: {bad[:12]}"
        if form == "bsag":
            info = st.info.cpu().numpy()
            finals = []
            for q in range(nb):
                c = min(int(info[nb + q]), st.k_blk)
                assert bool((st.sp_idx[q, q, c:] == INT32_MAX).all()), f"final padding block {q}"
                assert bool((st.sp_val[q, q, c:] == 0).all()), f"final padding values block {q}"
                finals.append(st.sp_idx[q, q, :c])
        else:
            finals = [st.sp_idx[q, q] for q in range(nb)]
        _check_member(st, finals, n)
        log(f"  step {t}: {len(done)} block indices x {len(want)} outputs match")
    del st, g, gen
    torch.cuda.empty_cache()


@pytest.mark.parametrize("workload,form,d", CASES, ids=[f"w{w}-{f}-d{d}" for w, f, d in CASES])
def test_full_size_every_block(workload, form, d):
    _run(workload, form, d)
