"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/spardl.h, its host-side schedule matches the paper's
examples and the oracle's schedule, and argument errors are reported before
anything is enqueued."""

import ctypes
import json
import os
import re

import pytest

from oracle import spardl_oracle as so

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2304_00737_amd", "libspardl.so")
HEADER = os.path.join(ROOT, "include", "spardl.h")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libspardl.so not built")


def _lib():
    lib = ctypes.CDLL(LIB)
    lib.spardl_srs_plan.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    lib.spardl_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, ctypes.c_int32]
    lib.spardl_workspace_bytes.restype = ctypes.c_size_t
    lib.spardl_strerror.restype = ctypes.c_char_p
    return lib


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+(spardl_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 8
    lib = _lib()
    for name in names:
        assert hasattr(lib, name), name


def test_srs_plan_matches_oracle_and_examples():
    lib = _lib()
    for P in range(1, 200):
        d = (ctypes.c_int32 * 32)()
        m = (ctypes.c_int32 * 32)()
        l = lib.spardl_srs_plan(P, d, m)
        steps = so.srs_schedule(P)
        assert l == len(steps) == so.num_steps(P)
        for st in steps:
            assert d[st.i - 1] == st.distance
            assert m[st.i - 1] == len(st.received_bag[0])
            for w in range(P):
                # the library's closed form: worker w receives blocks w .. w+m-1 from w - d
                assert list(st.received_bag[w]) == [(w + t) % P for t in range(m[st.i - 1])]
                assert st.source[w] == (w - d[st.i - 1]) % P
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "srs_examples_p6.json")))
    d = (ctypes.c_int32 * 32)()
    m = (ctypes.c_int32 * 32)()
    assert lib.spardl_srs_plan(6, d, m) == g["l"]
    assert [d[i] for i in range(3)] == [s["distance"] for s in g["steps"]]
    assert [m[i] for i in range(3)] == [s["sent_blocks"] for s in g["steps"]]
    assert lib.spardl_srs_plan(0, None, None) == -1


def test_workspace_bytes():
    lib = _lib()
    assert lib.spardl_workspace_bytes(1, 4, 100, 0) == 0          # k_blk < 1
    assert lib.spardl_workspace_bytes(1, 4, 100, 26) == 0         # k_blk > floor(n/P)
    assert lib.spardl_workspace_bytes(5, 4, 100, 3) == 0          # nworkers > P
    assert lib.spardl_workspace_bytes(1, 4, 2 ** 31, 3) == 0      # n >= 2^31
    a = lib.spardl_workspace_bytes(1, 8, 25_600_000, 32_000)
    b = lib.spardl_workspace_bytes(8, 8, 25_600_000, 32_000)
    assert 0 < a < b and b - a >= 7 * 25_600_000 * 8
    assert a % 256 == 0 and b % 256 == 0


def test_argument_errors_enqueue_nothing():
    """Invalid calls return a status before any HIP call (safe without a GPU)."""
    lib = _lib()
    p = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first
    null = ctypes.c_void_p(0)
    i64, i32, sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    EINVAL, ECAP = -1, -2
    # residual_add: NULL acc, ld < n, P > n
    assert lib.spardl_residual_add(null, i64(10), p, i64(10), i32(0), i32(1), i64(10), i32(0), i32(0), null, sz(0),
                                   null) == EINVAL
    assert lib.spardl_residual_add(p, i64(9), p, i64(10), i32(0), i32(1), i64(10), i32(0), i32(0), null, sz(0),
                                   null) == EINVAL
    assert lib.spardl_residual_add(p, i64(10), p, i64(10), i32(0), i32(1), i64(10), i32(11), i32(1), p, sz(1 << 20),
                                   null) == EINVAL
    assert lib.spardl_residual_add(p, i64(100), p, i64(100), i32(0), i32(2), i64(100), i32(4), i32(3), p, sz(16),
                                   null) == ECAP
    # with ws: k_blk outside [1, n / P]
    assert lib.spardl_residual_add(p, i64(100), p, i64(100), i32(0), i32(2), i64(100), i32(4), i32(26), p, sz(1 << 30),
                                   null) == EINVAL
    # the first worker of the call's rows: negative, or rows past P
    assert lib.spardl_residual_add(p, i64(100), p, i64(100), i32(-1), i32(1), i64(100), i32(4), i32(3), p,
                                   sz(1 << 30), null) == EINVAL
    assert lib.spardl_residual_add(p, i64(100), p, i64(100), i32(3), i32(2), i64(100), i32(4), i32(3), p,
                                   sz(1 << 30), null) == EINVAL
    assert lib.spardl_block_topk(p, i64(100), i32(3), i32(2), i64(100), i32(4), i32(3), i32(0), p, p, null, p,
                                 sz(1 << 30), null) == EINVAL
    assert lib.spardl_block_topk(p, i64(100), i32(-1), i32(1), i64(100), i32(4), i32(3), i32(0), p, p, null, p,
                                 sz(1 << 30), null) == EINVAL
    # block_topk: k_blk too large, flags unknown, nworkers > P, small workspace
    assert lib.spardl_block_topk(p, i64(100), i32(0), i32(1), i64(100), i32(4), i32(26), i32(0), p, p, null, p,
                                 sz(1 << 30), null) == EINVAL
    assert lib.spardl_block_topk(p, i64(100), i32(0), i32(1), i64(100), i32(4), i32(3), i32(4), p, p, null, p,
                                 sz(1 << 30), null) == EINVAL
    assert lib.spardl_block_topk(p, i64(100), i32(0), i32(5), i64(100), i32(4), i32(3), i32(0), p, p, null, p,
                                 sz(1 << 30), null) == EINVAL
    assert lib.spardl_block_topk(p, i64(100), i32(0), i32(1), i64(100), i32(4), i32(3), i32(0), p, p, null, p,
                                 sz(64), null) == ECAP
    # workspace_init: NULL, misaligned, too small, bad sizes
    lib.spardl_workspace_init.argtypes = [i32, i32, i64, i32, ctypes.c_void_p, sz, ctypes.c_void_p]
    assert lib.spardl_workspace_init(i32(1), i32(4), i64(100), i32(3), null, sz(1 << 30), null) == EINVAL
    assert lib.spardl_workspace_init(i32(1), i32(4), i64(100), i32(3), ctypes.c_void_p(0x1010), sz(1 << 30),
                                     null) == EINVAL
    assert lib.spardl_workspace_init(i32(1), i32(4), i64(100), i32(3), p, sz(64), null) == ECAP
    assert lib.spardl_workspace_init(i32(5), i32(4), i64(100), i32(3), p, sz(1 << 30), null) == EINVAL
    # a workspace that is not 256-byte aligned
    q = ctypes.c_void_p(0x1010)
    assert lib.spardl_block_topk(p, i64(100), i32(0), i32(1), i64(100), i32(4), i32(3), i32(0), p, p, null, q,
                                 sz(1 << 30), null) == EINVAL
    assert lib.spardl_sparse_merge_topk(p, p, i32(6), i64(600), i32(3), i32(1), p, p, p, q, sz(1 << 30),
                                        null) == EINVAL
    # merge: P < 2, round out of range, small workspace
    assert lib.spardl_sparse_merge_topk(p, p, i32(1), i64(100), i32(3), i32(1), p, p, p, p, sz(1 << 30), null) == EINVAL
    assert lib.spardl_sparse_merge_topk(p, p, i32(6), i64(600), i32(3), i32(4), p, p, p, p, sz(1 << 30), null) == EINVAL
    assert lib.spardl_sparse_merge_topk(p, p, i32(6), i64(600), i32(3), i32(0), p, p, p, p, sz(1 << 30), null) == EINVAL
    assert lib.spardl_sparse_merge_topk(p, p, i32(6), i64(600), i32(3), i32(1), p, p, p, p, sz(64), null) == ECAP
    # densify: n < P, NULL output, misaligned member bitmap
    assert lib.spardl_allgather_densify(p, p, i32(8), i64(7), i32(1), p, null, null) == EINVAL
    assert lib.spardl_allgather_densify(p, p, i32(2), i64(8), i32(1), null, null, null) == EINVAL
    assert lib.spardl_allgather_densify(p, p, i32(2), i64(8), i32(1), p, ctypes.c_void_p(0x1002), null) == EINVAL
    # residual_collect: missing per-step drop arrays for P > 1
    assert lib.spardl_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, p, null, null, null, null, p,
                                       sz(1 << 30), null) == EINVAL
    arr = (ctypes.c_void_p * 2)(0x1000, 0)
    assert lib.spardl_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, p, null, arr, arr, arr, p,
                                       sz(1 << 30), null) == EINVAL
    # residual_collect: without a member bitmap, sp_idx and an aligned ws are required
    ok3 = (ctypes.c_void_p * 2)(0x1000, 0x1000)
    assert lib.spardl_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, null, null, ok3, ok3, ok3, p,
                                       sz(1 << 30), null) == EINVAL
    assert lib.spardl_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, p, null, ok3, ok3, ok3, null,
                                       sz(1 << 30), null) == EINVAL
    assert lib.spardl_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, p, null, ok3, ok3, ok3, q,
                                       sz(1 << 30), null) == EINVAL
    assert lib.spardl_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, p, ctypes.c_void_p(0x1001),
                                       ok3, ok3, ok3, null, sz(0), null) == EINVAL
    # lazy_topk (P = 4, l = 2): round outside [0, l], rows outside [0, P), ld < n, small or misaligned ws
    big = sz(1 << 30)
    lt = lambda ld, w0, nw, rnd, ws, wsz, fl=0: lib.spardl_lazy_topk(p, i64(ld), i32(w0), i32(nw), i64(100), i32(4),
                                                                     i32(3), i32(rnd), i32(fl), p, p, ws, wsz, null)
    assert lt(100, 0, 1, 3, p, big) == EINVAL
    assert lt(100, 0, 1, -1, p, big) == EINVAL
    assert lt(100, 3, 2, 1, p, big) == EINVAL
    assert lt(100, -1, 1, 1, p, big) == EINVAL
    assert lt(100, 0, 0, 1, p, big) == EINVAL
    assert lt(99, 0, 1, 1, p, big) == EINVAL
    assert lt(100, 0, 1, 1, q, big) == EINVAL
    assert lt(100, 0, 1, 1, null, big) == EINVAL
    assert lt(100, 0, 1, 1, p, sz(64)) == ECAP
    assert lt(100, 0, 4, 1, p, big, 2) == EINVAL        # unknown flag
    assert lt(100, 1, 2, 1, p, big, 1) == EINVAL        # fused form on a row subset
    # lazy_receive: P = 1 has no steps; round outside [1, l]; NULL saved
    lr = lambda P_, rnd, saved, ws, wsz: lib.spardl_lazy_receive(p, i64(100), i32(P_), i64(100), i32(3), i32(rnd), p,
                                                                 p, saved, ws, wsz, null)
    assert lr(1, 1, p, null, sz(0)) == EINVAL
    assert lr(4, 0, p, null, sz(0)) == EINVAL
    assert lr(4, 3, p, null, sz(0)) == EINVAL
    assert lr(4, 1, null, null, sz(0)) == EINVAL
    assert lr(4, 1, p, q, big) == EINVAL                # misaligned workspace
    assert lr(4, 1, p, p, sz(64)) == ECAP               # workspace too small for the histograms
    # lazy_residual_collect: NULL or misaligned member, NULL saved with P > 1, k_blk too large
    assert lib.spardl_lazy_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, null, p, null) == EINVAL
    assert lib.spardl_lazy_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, ctypes.c_void_p(0x1002), p,
                                            null) == EINVAL
    assert lib.spardl_lazy_residual_collect(p, i64(100), i32(4), i64(100), i32(3), p, p, null, null) == EINVAL
    assert lib.spardl_lazy_residual_collect(p, i64(100), i32(4), i64(100), i32(26), p, p, p, null) == EINVAL
    # R-SAG: d not a power of 2 or not dividing P, t out of range, small workspace, missing drop arrays
    lib.spardl_rsag_workspace_bytes.argtypes = [i32, i32, i64, i32]
    lib.spardl_rsag_workspace_bytes.restype = sz
    assert lib.spardl_rsag_workspace_bytes(i32(12), i32(3), i64(1200), i32(5)) == 0
    assert lib.spardl_rsag_workspace_bytes(i32(12), i32(8), i64(1200), i32(5)) == 0
    assert lib.spardl_rsag_workspace_bytes(i32(8), i32(1), i64(1200), i32(5)) == 0
    assert lib.spardl_rsag_workspace_bytes(i32(8), i32(4), i64(1200), i32(601)) == 0
    assert lib.spardl_rsag_workspace_bytes(i32(8), i32(4), i64(1200), i32(600)) > 0
    rm = lambda t, ws, wsz: lib.spardl_rsag_merge_topk(p, p, i32(8), i32(4), i64(1200), i32(5), i32(t), p, p, p,
                                                       ws, wsz, null)
    assert rm(2, p, big) == EINVAL
    assert rm(-1, p, big) == EINVAL
    assert rm(0, q, big) == EINVAL
    assert rm(0, p, sz(64)) == ECAP
    assert lib.spardl_rsag_merge_topk(p, p, i32(8), i32(3), i64(1200), i32(5), i32(0), p, p, p, p, big,
                                      null) == EINVAL
    one = (ctypes.c_void_p * 2)(0x1000, 0)
    assert lib.spardl_rsag_residual(p, i64(1200), i32(8), i32(4), i64(1200), i32(5), p, one, one, one,
                                    null) == EINVAL
    assert lib.spardl_rsag_residual(p, i64(1200), i32(8), i32(4), i64(1200), i32(5), null, ok3, ok3, ok3,
                                    null) == EINVAL
    assert lib.spardl_rsag_residual(p, i64(1199), i32(8), i32(4), i64(1200), i32(5), p, ok3, ok3, ok3,
                                    null) == EINVAL
    lib.spardl_rsag_workspace_init.argtypes = [i32, i32, i64, i32, ctypes.c_void_p, sz, ctypes.c_void_p]
    assert lib.spardl_rsag_workspace_init(i32(8), i32(4), i64(1200), i32(5), q, big, null) == EINVAL
    assert lib.spardl_rsag_workspace_init(i32(8), i32(4), i64(1200), i32(5), p, sz(64), null) == ECAP
    # B-SAG: d not dividing P, k_blk too large for a team block, small or misaligned workspace
    lib.spardl_bsag_workspace_bytes.argtypes = [i32, i32, i64, i32]
    lib.spardl_bsag_workspace_bytes.restype = sz
    assert lib.spardl_bsag_workspace_bytes(i32(14), i32(4), i64(1400), i32(5)) == 0
    assert lib.spardl_bsag_workspace_bytes(i32(14), i32(1), i64(1400), i32(5)) == 0
    assert lib.spardl_bsag_workspace_bytes(i32(14), i32(7), i64(1400), i32(701)) == 0
    assert lib.spardl_bsag_workspace_bytes(i32(14), i32(7), i64(1400), i32(700)) > 0
    bx = lambda P_, d_, ws, wsz: lib.spardl_bsag_exchange(p, p, i32(P_), i32(d_), i64(1400), i32(5), p, p, p, null,
                                                          ws, wsz, null)
    assert bx(14, 4, p, big) == EINVAL
    assert bx(14, 7, q, big) == EINVAL
    assert bx(14, 7, p, sz(64)) == ECAP
    assert lib.spardl_bsag_residual(p, i64(1400), i32(14), i32(7), i64(1400), i32(5), null, p, p, p,
                                    null) == EINVAL
    assert lib.spardl_bsag_residual(p, i64(1400), i32(14), i32(7), i64(1400), i32(5), p, null, p, p,
                                    null) == EINVAL
    lib.spardl_bsag_workspace_init.argtypes = [i32, i32, i64, i32, ctypes.c_void_p, sz, ctypes.c_void_p]
    assert lib.spardl_bsag_workspace_init(i32(14), i32(7), i64(1400), i32(5), q, big, null) == EINVAL
    assert lib.spardl_bsag_workspace_init(i32(14), i32(7), i64(1400), i32(5), p, sz(64), null) == ECAP
    # team calls: d not dividing P, k_blk too large for a team block, round out of range, small workspace
    lib.spardl_team_workspace_bytes.argtypes = [i32, i32, i64, i32]
    lib.spardl_team_workspace_bytes.restype = sz
    assert lib.spardl_team_workspace_bytes(i32(12), i32(5), i64(1200), i32(5)) == 0
    assert lib.spardl_team_workspace_bytes(i32(12), i32(4), i64(1200), i32(401)) == 0
    assert lib.spardl_team_workspace_bytes(i32(12), i32(4), i64(1200), i32(400)) > 0
    tm = lambda rnd, wsz: lib.spardl_team_merge_topk(p, p, i32(12), i32(4), i64(1200), i32(5), i32(rnd), p, p, p, p,
                                                     wsz, null)
    assert tm(0, big) == EINVAL
    assert tm(3, big) == EINVAL          # Q = 3: two steps
    assert tm(1, sz(64)) == ECAP
    assert lib.spardl_team_block_topk(p, i64(1200), i32(12), i32(4), i64(1200), i32(5), i32(2), p, p, null, p, big,
                                      null) == EINVAL
    assert lib.spardl_team_residual_add(p, i64(1199), p, i64(1200), i32(12), i32(4), i64(1200), i32(5), p, big,
                                        null) == EINVAL
    # residual add with the previous step's collection (P = 4: two SRS steps): member, local_idx, ws and
    # every drop pointer required; rows inside [0, P); a workspace too small
    ac = lambda ld, w0, nw, li, mem, a, ws, wsz: lib.spardl_residual_add_collect(
        p, i64(ld), p, i64(100), i32(w0), i32(nw), i64(100), i32(4), i32(3), li, mem, a, a, a, ws, wsz, null)
    assert ac(100, 0, 4, p, null, ok3, p, big) == EINVAL
    assert ac(100, 0, 4, null, p, ok3, p, big) == EINVAL
    assert ac(100, 0, 4, p, ctypes.c_void_p(0x1002), ok3, p, big) == EINVAL
    assert ac(100, 0, 4, p, p, arr, p, big) == EINVAL
    assert ac(100, 0, 4, p, p, null, p, big) == EINVAL
    assert ac(100, 0, 4, p, p, ok3, null, big) == EINVAL
    assert ac(100, 0, 4, p, p, ok3, q, big) == EINVAL
    assert ac(99, 0, 4, p, p, ok3, p, big) == EINVAL
    assert ac(100, 2, 3, p, p, ok3, p, big) == EINVAL
    assert ac(100, -1, 1, p, p, ok3, p, big) == EINVAL
    assert ac(100, 0, 4, p, p, ok3, p, sz(64)) == ECAP
    # the drop-tile index (P = 4: two SRS steps): aligned ws, rows inside [0, P), every drop pointer
    ci = lambda w0, nw, a, ws, wsz: lib.spardl_residual_collect_index(i32(w0), i32(nw), i64(100), i32(4), i32(3),
                                                                      a, a, ws, wsz, null)
    assert ci(0, 4, ok3, null, big) == EINVAL
    assert ci(0, 4, ok3, q, big) == EINVAL
    assert ci(0, 4, arr, p, big) == EINVAL
    assert ci(0, 4, null, p, big) == EINVAL
    assert ci(1, 4, ok3, p, big) == EINVAL
    assert ci(0, 0, ok3, p, big) == EINVAL
    assert ci(0, 4, ok3, p, sz(64)) == ECAP
    # team residual collect (Q = 3: two rounds of drops): member required and aligned, every drop pointer, d | P
    tc = lambda d_, mem, a: lib.spardl_team_residual_collect(p, i64(1200), i32(12), i32(d_), i64(1200), i32(5), p,
                                                             mem, a, a, a, null)
    assert tc(4, null, ok3) == EINVAL
    assert tc(4, ctypes.c_void_p(0x1002), ok3) == EINVAL
    assert tc(4, p, arr) == EINVAL
    assert tc(4, p, null) == EINVAL
    assert tc(5, p, ok3) == EINVAL
    # the workspace-free SRS step: NULL err, P < 2, round out of range; a step whose scratch exceeds the
    # library's static array is refused before any GPU call (P = 32, k_blk = 46875: 512 pairs of 23 slots)
    na = lambda P_, n_, kb_, rnd, err: lib.spardl_sparse_merge_topk_noalloc(p, p, i32(P_), i64(n_), i32(kb_), i32(rnd),
                                                                           p, p, p, err, null)
    assert na(8, 800, 5, 1, null) == EINVAL
    assert na(1, 800, 5, 1, p) == EINVAL
    assert na(8, 800, 5, 0, p) == EINVAL
    assert na(8, 800, 5, 4, p) == EINVAL
    assert na(8, 800, 101, 1, p) == EINVAL
    assert na(32, 1_500_000_000, 46875, 1, p) == ECAP
    assert na(16, 110_000_000, 68750, 1, p) == ECAP
    for s in (0, -1, -2, -3, 7):
        assert lib.spardl_strerror(s)


def test_ws_layout_mirror():
    """The GPU tests read workspace words through a Python mirror of the
    layout; its total must equal the library's workspace size."""
    from tests.gpu_util import ws_layout
    lib = _lib()
    al = lambda x: (x + 255) & ~255
    # (the last three have blocks of 3357, 8423 and 22889 add tiles: 8, 32 and 32 histogram copies)
    for P, n, kb in [(1, 5000, 7), (4, 1 << 20, 2622), (5, 6000, 1200), (8, 25_600_000, 32_000), (16, 65536, 41),
                     (12, 60000, 50), (3, 100003, 33334), (16, 110_000_000, 68_750), (8, 138_000_000, 86_250),
                     (32, 1_500_000_000, 46_875)]:
        L = ws_layout(P, n, kb, 0)
        assert L["fixed_end"] + 3 * al(L["cand_entries"] * 4) == lib.spardl_workspace_bytes(P, P, n, kb), (P, n, kb)
