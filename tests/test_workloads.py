"""The seeded synthetic-gradient generator (input plumbing shared by the oracle
and the GPU path): determinism, element addressability, the math it relies
on, and the documented workload shapes."""

import math
import os

import numpy as np
import pytest

from paper_2304_00737_amd import workloads as W

pytestmark = pytest.mark.skipif(not os.path.exists(W.LIB_PATH), reason="libgradgen.so not built")


def test_config_shapes():
    # (P, n, k, k/P) of the five workloads; k = ceil(rho n), k/P rounded up
    want = {1: (4, 1 << 20, 10486, 2622), 2: (8, 25_600_000, 256_000, 32_000),
            3: (8, 138_000_000, 690_000, 86_250), 4: (16, 110_000_000, 1_100_000, 68_750),
            5: (32, 1_500_000_000, 1_500_000, 46_875)}
    for c, (P, n, k, kb) in want.items():
        wl = W.config(c)
        assert (wl.P, wl.n, wl.k, wl.k_blk) == (P, n, k, kb)
        assert sum(wl.seg_len) == n and all(s > 0 for s in wl.seg_len)
    assert len(W.config(2).seg_len) == 160
    wl3 = W.config(3)
    assert len(wl3.seg_len) == 16 and wl3.seg_len[13] == 102_760_448
    assert len(W.config(4).seg_len) == 200 and W.config(4).zero_prob == 0.2
    assert W.config(5).seg_len == (31_250_000,) * 48


def test_deterministic_and_addressable():
    wl = W.config(4)
    a = W.gradient(wl, 2, 5, 1_000_000, 50_000)
    b = W.gradient(wl, 2, 5, 1_000_000, 50_000)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    c = W.gradient(wl, 2, 5, 999_000, 60_000)[1000:51000]
    assert np.array_equal(a.view(np.uint32), c.view(np.uint32))
    d = W.gradient(wl, 2, 6, 1_000_000, 50_000)       # another worker differs
    assert not np.array_equal(a, d)


def test_log_matches_libm():
    lib = W._load()
    rng = np.random.default_rng(0)
    xs = np.concatenate([rng.uniform(1e-12, 1.0, 2000), 10.0 ** rng.uniform(-300, 300, 2000)])
    for x in xs:
        got, want = lib.gg_log_host(float(x)), math.log(float(x))
        assert abs(got - want) <= 4e-16 * max(1.0, abs(want))


def test_distributions():
    n = 400_000
    normal = W.Workload(9, "t", 1, n, (1, 100), 1, "normal", (n,), (1.0,))
    g = W.gradient(normal, 1, 0).astype(np.float64)
    assert abs(g.mean()) < 0.01 and abs(g.std() - 1.0) < 0.01
    assert abs(np.mean(np.abs(g) > 1.959964) - 0.05) < 0.003
    lap = W.Workload(9, "t", 1, n, (1, 100), 1, "laplace", (n,), (2.0,))
    g = W.gradient(lap, 1, 0).astype(np.float64)
    assert abs(np.mean(np.abs(g)) - 2.0) < 0.02          # E|X| = b
    t3 = W.Workload(9, "t", 1, n, (1, 100), 1, "student_t3", (n,), (1.0,), zero_prob=0.2)
    g = W.gradient(t3, 1, 0).astype(np.float64)
    assert abs(np.mean(g == 0.0) - 0.2) < 0.005
    nz = g[g != 0.0]
    assert abs(np.mean(np.abs(nz) > 3.182446) - 0.05) < 0.003   # t(3) two-sided 5% point


def test_segment_scales_apply():
    wl = W.config(2)
    starts = wl.seg_start
    s = int(np.argmax(wl.seg_len))
    g = W.gradient(wl, 1, 0, int(starts[s]), int(wl.seg_len[s])).astype(np.float64)
    assert abs(g.std() / wl.seg_scale[s] - 1.0) < 0.01
