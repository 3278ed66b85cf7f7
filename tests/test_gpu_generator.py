"""The device build of the input generator gives the host generator's bits.

The largest workload creates its per-worker gradients on the GPU; its parity
checks regenerate the same slices on the host for the oracle, so the two
builds must agree exactly, for every distribution, across segment
boundaries and for both steps and any worker.
"""

import numpy as np
import pytest

from tests.conftest import gpu_available
from tests.gpu_util import log

pytestmark = pytest.mark.gpu

if gpu_available():
    import torch
    from paper_2304_00737_amd import workloads as W


@pytest.mark.parametrize("cfg_id", [1, 2, 3, 4, 5])
def test_device_generator_matches_host(cfg_id):
    wl = W.config(cfg_id)
    gen = W.DeviceGenerator(wl)
    starts = wl.seg_start
    slices = [(0, 1 << 18), (wl.n - 4099, 4099)]
    for s in (1, len(starts) // 2, len(starts) - 2):   # around segment boundaries
        x = int(starts[s])
        slices.append((max(0, x - 2000), min(4000, wl.n - max(0, x - 2000))))
    log(f"generator {wl.name}: {len(slices)} slices")
    for step in (1, wl.steps):
        for worker in (0, wl.P - 1):
            for x0, cnt in slices:
                dev = torch.empty(cnt, dtype=torch.float32, device="cuda")
                gen.fill(dev, step, worker, x0)
                host = W.gradient(wl, step, worker, x0, cnt)
                got = dev.cpu().numpy()
                bad = np.nonzero(got.view(np.uint32) != host.view(np.uint32))[0]
                assert bad.size == 0, (f"step {step} worker {worker} x {x0 + bad[0]}: "
                                       f"device {got[bad[0]]!r} host {host[bad[0]]!r}")
