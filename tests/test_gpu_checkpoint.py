"""Checkpoint and resume of the only state a step carries to the next:
Algorithm 1's residual xi (and, for B-SAG, Algorithm 2's controller).  Three
consecutive steps must equal one step, a checkpoint copied to host memory
and loaded into fresh objects, and two more steps, byte for byte."""

import numpy as np
import pytest

from tests.conftest import gpu_available
from tests.gpu_util import log

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    from paper_2304_00737_amd import spardl
    from paper_2304_00737_amd import workloads as W

P, N, KB = 6, 60000, 90


def _make(form):
    if form in ("eager", "eager_fc"):   # eager_fc: each collection inside the next step's add
        return spardl.SparDLStep(P, N, KB, fuse_collect=form == "eager_fc")
    if form == "lazy":
        return spardl.SparDLLazyStep(P, N, KB)
    if form == "rsag":
        return spardl.SparDLSagStep(8, 2, N, KB)
    return spardl.SparDLSagStep(P, 3, N, KB, bruck=True)


def _outputs(st):
    if hasattr(st, "flush"):
        st.flush()   # the last step's pending collection, if any
    t = [st.acc, st.dense, st.sp_idx, st.sp_val]
    if hasattr(st, "info"):
        t.append(st.info)
    return [x.cpu().numpy().tobytes() for x in t]


@pytest.mark.parametrize("form", ["eager", "eager_fc", "lazy", "rsag", "bsag"])
def test_resume_from_checkpoint(form):
    log(f"checkpoint and resume: {form}")
    rows = 8 if form == "rsag" else P
    grads = [torch.from_numpy(W.small_rows("normal", rows, N, 700 + t)).cuda() for t in range(3)]
    a = _make(form)
    for g in grads:
        a.step(g)
    torch.cuda.synchronize()
    want = _outputs(a)
    b = _make(form)
    b.step(grads[0])
    ckpt = b.state_dict()
    assert all(v.device.type == "cpu" for v in ckpt.values())
    del b
    c = _make(form)
    c.load_state_dict(ckpt)
    for g in grads[1:]:
        c.step(g)
    torch.cuda.synchronize()
    got = _outputs(c)
    for i, (x, y) in enumerate(zip(got, want)):
        assert x == y, f"output {i} differs after resuming"
    log("  resumed run equals the continuous one")
