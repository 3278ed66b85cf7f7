"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare with the oracle bit for bit."""

from __future__ import annotations

import sys

import numpy as np

from oracle import spardl_oracle as so


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def bits(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32)).view(np.uint32)


def assert_bits_equal(got, want, what: str) -> None:
    g, w = bits(got), bits(want)
    if g.shape != w.shape or not np.array_equal(g, w):
        bad = np.nonzero(g != w)[0] if g.shape == w.shape else None
        first = int(bad[0]) if bad is not None and len(bad) else -1
        raise AssertionError(f"{what}: shapes {g.shape} vs {w.shape}; {0 if bad is None else len(bad)} "
                             f"mismatches, first at {first}: got {g.view(np.float32)[first] if first >= 0 else None} "
                             f"want {w.view(np.float32)[first] if first >= 0 else None}")


def assert_idx_equal(got, want, what: str) -> None:
    g = np.asarray(got, dtype=np.int64)
    w = np.asarray(want, dtype=np.int64)
    if g.shape != w.shape or not np.array_equal(g, w):
        raise AssertionError(f"{what}: index mismatch (shapes {g.shape} vs {w.shape})")


def check_ws(st) -> None:
    from paper_2304_00737_amd import spardl
    e = spardl.ws_error(st.ws)
    assert e == 0, f"workspace error word {e}"


def compare_step(st, res, P: int, n: int, kb: int, blocks=None, acc_host=None) -> None:
    """Compare the GPU state after one step with an oracle SparDLStepResult."""
    blocks = list(range(P)) if blocks is None else list(blocks)
    bounds = so.block_bounds(n, P)
    sp_idx = st.sp_idx.cpu().numpy()
    sp_val = st.sp_val.cpu().numpy()
    local = st.local_idx.cpu().numpy()
    for w in range(P):
        for b in blocks:
            li, lv = res.local[(w, b)]
            assert_idx_equal(local[w, b], li, f"local_idx w={w} b={b}")
            si, sv = res.S[(w, b)]
            assert_idx_equal(sp_idx[w, b], si, f"sp_idx w={w} b={b}")
            assert_bits_equal(sp_val[w, b], sv, f"sp_val w={w} b={b}")
    for i, m in enumerate(st.bags, start=1):
        di = st.drop_idx[i - 1].cpu().numpy()
        dv = st.drop_val[i - 1].cpu().numpy()
        dc = st.drop_cnt[i - 1].cpu().numpy()
        for w in range(P):
            for t in range(m):
                b = (w + t) % P
                if b not in blocks:
                    continue
                oi, ov = res.drops[(i, w, b)]
                c = int(dc[w, t])
                assert c == len(oi), f"drop count step {i} w={w} b={b}: {c} vs {len(oi)}"
                assert_idx_equal(di[w, t, :c], oi, f"drop idx step {i} w={w} b={b}")
                assert_bits_equal(dv[w, t, :c], ov, f"drop val step {i} w={w} b={b}")
    n_drops = sum(1 for (i, w, b) in res.drops if b in blocks)
    assert n_drops == sum(P * m for m in st.bags) * len(blocks) // P
    dense = st.dense
    for b in blocks:
        got = dense[bounds[b]:bounds[b + 1]].cpu().numpy()
        assert_bits_equal(got, res.dense[b], f"dense block {b}")
    for w in range(P):
        for b in blocks:
            got = st.acc[w, bounds[b]:bounds[b + 1]].cpu().numpy()
            assert_bits_equal(got, res.residual[(w, b)], f"residual w={w} b={b}")
