"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare with the oracle bit for bit."""

from __future__ import annotations

import sys

import numpy as np
import torch

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


def compare_step(st, res, P: int, n: int, kb: int, blocks=None, acc_host=None, residual=True) -> None:
    """Compare the GPU state after one step with an oracle SparDLStepResult
    (residual=False: not acc, whose collection is still pending)."""
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
    for w in range(P if residual else 0):
        for b in blocks:
            got = st.acc[w, bounds[b]:bounds[b + 1]].cpu().numpy()
            assert_bits_equal(got, res.residual[(w, b)], f"residual w={w} b={b}")
    if getattr(st, "fused", False):   # densify also wrote the membership bitmap of I
        words = st.member.cpu().numpy()
        bits = np.unpackbits(words.view(np.uint8), bitorder="little").astype(bool)
        assert not bits[n:].any(), "member bits at or above n"
        for b in blocks:
            want = np.zeros(bounds[b + 1] - bounds[b], bool)
            want[np.asarray(res.final[b][0], np.int64) - bounds[b]] = True
            assert np.array_equal(bits[bounds[b]:bounds[b + 1]], want), f"member bits block {b}"


def ws_layout(P: int, n: int, kb: int, ws_bytes: int) -> dict:
    """The binding's mirror of the workspace layout (imported on use: the
    binding needs the built library)."""
    from paper_2304_00737_amd.spardl import ws_layout as _ws_layout
    return _ws_layout(P, n, kb, ws_bytes)


def ws_spec_ok(st) -> list:
    """Per (worker, block): did the last block top-k use the fused add's candidates?"""
    L = ws_layout(st.P, st.n, st.k_blk, st.ws.numel())
    words = st.ws[L["state"]:L["state"] + st.P * st.P * 16 * 4].view(torch.int32).cpu().numpy()
    return [bool(words[u * 16 + 7]) for u in range(st.P * st.P)]


def compare_lazy_step(st, res, P: int, n: int, kb: int, blocks=None) -> None:
    """Compare the GPU state after one lazy step with an oracle LazyStepResult:
    every worker's selection of every listed block, the dense update, the
    membership bitmap of I and the new residuals, bit for bit."""
    blocks = list(range(P)) if blocks is None else list(blocks)
    bounds = so.block_bounds(n, P)
    sp_idx = st.sp_idx[:, blocks].cpu().numpy()
    sp_val = st.sp_val[:, blocks].cpu().numpy()
    for w in range(P):
        for j, b in enumerate(blocks):
            si, sv = res.sel[(w, b)]
            assert_idx_equal(sp_idx[w, j], si, f"selection w={w} b={b} (sent at step {res.sent_at[(w, b)]})")
            assert_bits_equal(sp_val[w, j], sv, f"selection value w={w} b={b}")
    words = st.member.cpu().numpy()
    mbits = np.unpackbits(words.view(np.uint8), bitorder="little").astype(bool)
    assert not mbits[n:].any(), "member bits at or above n"
    for b in blocks:
        got = st.dense[bounds[b]:bounds[b + 1]].cpu().numpy()
        assert_bits_equal(got, res.dense[b], f"dense block {b}")
        want = np.zeros(bounds[b + 1] - bounds[b], bool)
        want[np.asarray(res.final[b][0], np.int64) - bounds[b]] = True
        assert np.array_equal(mbits[bounds[b]:bounds[b + 1]], want), f"member bits block {b}"
    for w in range(P):
        for b in blocks:
            got = st.acc[w, bounds[b]:bounds[b + 1]].cpu().numpy()
            assert_bits_equal(got, res.residual[(w, b)], f"residual w={w} b={b}")


def compare_sag_step(st, res, blocks=None) -> None:
    """Compare the GPU state after one R-SAG step with an oracle SagStepResult:
    local selections, the sparse state of every block, the SRS drops inside
    every team, the drops of every exchange, the dense update, the bitmap of I
    and the residuals, bit for bit."""
    P, d, Q, n = st.P, st.d, st.Q, st.n
    blocks = list(range(Q)) if blocks is None else list(blocks)
    bounds = so.block_bounds(n, Q)
    sp_idx, sp_val = st.sp_idx.cpu().numpy(), st.sp_val.cpu().numpy()
    local = st.local_idx.cpu().numpy()
    for w in range(P):
        for b in blocks:
            assert_idx_equal(local[w, b], res.local[(w, b)][0], f"local_idx w={w} b={b}")
            si, sv = res.S[(w, b)]
            assert_idx_equal(sp_idx[w, b], si, f"sp_idx w={w} b={b}")
            assert_bits_equal(sp_val[w, b], sv, f"sp_val w={w} b={b}")
    for i, m in enumerate(st.bags, start=1):
        di, dv, dc = (x[i - 1].cpu().numpy() for x in (st.drop_idx, st.drop_val, st.drop_cnt))
        for w in range(P):
            q = w % Q
            for t in range(m):
                b = (q + t) % Q
                if b not in blocks:
                    continue
                oi, ov = res.drops[(i, w, b)]
                c = int(dc[w, t])
                assert c == len(oi), f"team drop count step {i} w={w} b={b}"
                assert_idx_equal(di[w, t, :c], oi, f"team drop idx step {i} w={w} b={b}")
                assert_bits_equal(dv[w, t, :c], ov, f"team drop val step {i} w={w} b={b}")
    for t in range(st.steps):
        si, sv, sc = (x[t].cpu().numpy() for x in (st.sag_idx, st.sag_val, st.sag_cnt))
        for p in range(len(sc)):
            j, q = divmod(p, Q)
            if q not in blocks:
                continue
            low = j & ((1 << t) - 1)
            X = ((j >> t) << (t + 1)) | low
            oi, ov = res.sag_drops[(t, X * Q + q)]
            c = int(sc[p])
            assert c == len(oi), f"exchange {t} drop count pair {p}"
            assert_idx_equal(si[p, :c], oi, f"exchange {t} drop idx pair {p}")
            assert_bits_equal(sv[p, :c], ov, f"exchange {t} drop val pair {p}")
    words = st.member.cpu().numpy()
    mbits = np.unpackbits(words.view(np.uint8), bitorder="little").astype(bool)
    assert not mbits[n:].any(), "member bits at or above n"
    for b in blocks:
        assert_bits_equal(st.dense[bounds[b]:bounds[b + 1]].cpu().numpy(), res.dense[b], f"dense block {b}")
        want = np.zeros(bounds[b + 1] - bounds[b], bool)
        want[np.asarray(res.final[b][0], np.int64) - bounds[b]] = True
        assert np.array_equal(mbits[bounds[b]:bounds[b + 1]], want), f"member bits block {b}"
    for w in range(P):
        for b in blocks:
            got = st.acc[w, bounds[b]:bounds[b + 1]].cpu().numpy()
            assert_bits_equal(got, res.residual[(w, b)], f"residual w={w} b={b}")


def compare_bsag_step(st, res, blocks=None) -> None:
    """Compare the GPU state after one B-SAG step with an oracle BsagStepResult:
    local selections, every worker's block state after its team's SRS, the
    SRS drops, the controller's counts and union sizes, every worker's top-h
    drops, the final blocks (sentinel-padded in sp[q][q]), the dense update,
    the bitmap of I and the residuals, bit for bit."""
    P, d, Q, n, L = st.P, st.d, st.Q, st.n, st.k_blk
    blocks = list(range(Q)) if blocks is None else list(blocks)
    bounds = so.block_bounds(n, Q)
    sp_idx, sp_val = st.sp_idx.cpu().numpy(), st.sp_val.cpu().numpy()
    local = st.local_idx.cpu().numpy()
    for w in range(P):
        for b in blocks:
            assert_idx_equal(local[w, b], res.local[(w, b)][0], f"local_idx w={w} b={b}")
            if w == b:           # team 0's holder of block b: the final block
                fi, fv = res.final[b]
                c = len(fi)
                assert_idx_equal(sp_idx[w, b, :c], fi, f"final idx block {b}")
                assert_bits_equal(sp_val[w, b, :c], fv, f"final val block {b}")
                assert (sp_idx[w, b, c:] == np.iinfo(np.int32).max).all(), f"final padding block {b}"
                assert (sp_val[w, b, c:] == 0).all(), f"final padding values block {b}"
                continue
            si, sv = res.S[(w, b)]
            assert_idx_equal(sp_idx[w, b], si, f"sp_idx w={w} b={b}")
            assert_bits_equal(sp_val[w, b], sv, f"sp_val w={w} b={b}")
    for i, m in enumerate(st.bags, start=1):
        di, dv, dc = (x[i - 1].cpu().numpy() for x in (st.drop_idx, st.drop_val, st.drop_cnt))
        for w in range(P):
            q = w % Q
            for t in range(m):
                b = (q + t) % Q
                if b not in blocks:
                    continue
                oi, ov = res.drops[(i, w, b)]
                c = int(dc[w, t])
                assert c == len(oi), f"team drop count step {i} w={w} b={b}"
                assert_idx_equal(di[w, t, :c], oi, f"team drop idx step {i} w={w} b={b}")
                assert_bits_equal(dv[w, t, :c], ov, f"team drop val step {i} w={w} b={b}")
    info = st.info.cpu().numpy()
    th_i, th_v, th_c = st.toph_idx.cpu().numpy(), st.toph_val.cpu().numpy(), st.toph_cnt.cpu().numpy()
    for q in blocks:
        assert int(info[q]) == res.h[q], f"top-h count block {q}: {int(info[q])} vs {res.h[q]}"
        assert int(info[Q + q]) == len(res.union[q][0]), f"union size block {q}"
        for tau in range(d):
            w = tau * Q + q
            oi, ov = res.drop_h[w]
            c = int(th_c[w])
            assert c == len(oi), f"top-h drop count w={w}"
            assert_idx_equal(th_i[w, :c], oi, f"top-h drop idx w={w}")
            assert_bits_equal(th_v[w, :c], ov, f"top-h drop val w={w}")
    words = st.member.cpu().numpy()
    mbits = np.unpackbits(words.view(np.uint8), bitorder="little").astype(bool)
    assert not mbits[n:].any(), "member bits at or above n"
    for b in blocks:
        assert_bits_equal(st.dense[bounds[b]:bounds[b + 1]].cpu().numpy(), res.dense[b], f"dense block {b}")
        want = np.zeros(bounds[b + 1] - bounds[b], bool)
        want[np.asarray(res.final[b][0], np.int64) - bounds[b]] = True
        assert np.array_equal(mbits[bounds[b]:bounds[b + 1]], want), f"member bits block {b}"
    for w in range(P):
        for b in blocks:
            got = st.acc[w, bounds[b]:bounds[b + 1]].cpu().numpy()
            assert_bits_equal(got, res.residual[(w, b)], f"residual w={w} b={b}")
