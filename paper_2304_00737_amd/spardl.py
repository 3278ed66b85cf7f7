"""Thin Python binding of libspardl.so (argument marshalling only).

Every function has the name of the C entry point in include/spardl.h without
the ``spardl_`` prefix, takes torch tensors for device buffers (torch is used
for device memory and streams only), checks the returned status and raises
SpardlError on failure.  All compute runs in the HIP kernels of libspardl.so;
there is no fallback: if the library is missing, importing this module fails.
"""

from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libspardl.so")

OK, EINVAL, ECAPACITY, EDEVICE = 0, -1, -2, -3
TOPK_HIST_READY = 1
WS_ERR_LOOKBACK = 1
WS_ERR_COUNT = 2

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built (run __graft_entry__.build()); "
                      "there is no fallback implementation")

_lib = ctypes.CDLL(LIB_PATH)
_p, _i32, _i64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t

_lib.spardl_strerror.argtypes = [ctypes.c_int]
_lib.spardl_strerror.restype = ctypes.c_char_p
_lib.spardl_srs_plan.argtypes = [_i32, _p, _p]
_lib.spardl_srs_plan.restype = ctypes.c_int
_lib.spardl_workspace_bytes.argtypes = [_i32, _i32, _i64, _i32]
_lib.spardl_workspace_bytes.restype = _sz
_lib.spardl_workspace_init.argtypes = [_i32, _i32, _i64, _i32, _p, _sz, _p]
_lib.spardl_workspace_init.restype = ctypes.c_int
_lib.spardl_residual_add.argtypes = [_p, _i64, _p, _i64, _i32, _i32, _i64, _i32, _i32, _p, _sz, _p]
_lib.spardl_residual_add_collect.argtypes = [_p, _i64, _p, _i64, _i32, _i32, _i64, _i32, _i32, _p, _p, _p, _p, _p, _p,
                                             _sz, _p]
_lib.spardl_residual_collect_index.argtypes = [_i32, _i32, _i64, _i32, _i32, _p, _p, _p, _sz, _p]
_lib.spardl_block_topk.argtypes = [_p, _i64, _i32, _i32, _i64, _i32, _i32, _i32, _p, _p, _p, _p, _sz, _p]
_lib.spardl_sparse_merge_topk.argtypes = [_p, _p, _i32, _i64, _i32, _i32, _p, _p, _p, _p, _sz, _p]
_lib.spardl_sparse_merge_topk_noalloc.argtypes = [_p, _p, _i32, _i64, _i32, _i32, _p, _p, _p, _p, _p]
_lib.spardl_allgather_densify.argtypes = [_p, _p, _i32, _i64, _i32, _p, _p, _p]
_lib.spardl_residual_collect.argtypes = [_p, _i64, _i32, _i64, _i32, _p, _p, _p, _p, _p, _p, _p, _sz, _p]
_lib.spardl_lazy_topk.argtypes = [_p, _i64, _i32, _i32, _i64, _i32, _i32, _i32, _i32, _p, _p, _p, _sz, _p]
_lib.spardl_lazy_receive.argtypes = [_p, _i64, _i32, _i64, _i32, _i32, _p, _p, _p, _p, _sz, _p]
_lib.spardl_lazy_residual_collect.argtypes = [_p, _i64, _i32, _i64, _i32, _p, _p, _p, _p]
_lib.spardl_rsag_workspace_bytes.argtypes = [_i32, _i32, _i64, _i32]
_lib.spardl_rsag_workspace_bytes.restype = _sz
_lib.spardl_rsag_workspace_init.argtypes = [_i32, _i32, _i64, _i32, _p, _sz, _p]
_lib.spardl_rsag_merge_topk.argtypes = [_p, _p, _i32, _i32, _i64, _i32, _i32, _p, _p, _p, _p, _sz, _p]
_lib.spardl_rsag_residual.argtypes = [_p, _i64, _i32, _i32, _i64, _i32, _p, _p, _p, _p, _p]
_lib.spardl_team_workspace_bytes.argtypes = [_i32, _i32, _i64, _i32]
_lib.spardl_team_workspace_bytes.restype = _sz
_lib.spardl_team_workspace_init.argtypes = [_i32, _i32, _i64, _i32, _p, _sz, _p]
_lib.spardl_team_residual_add.argtypes = [_p, _i64, _p, _i64, _i32, _i32, _i64, _i32, _p, _sz, _p]
_lib.spardl_team_block_topk.argtypes = [_p, _i64, _i32, _i32, _i64, _i32, _i32, _p, _p, _p, _p, _sz, _p]
_lib.spardl_team_merge_topk.argtypes = [_p, _p, _i32, _i32, _i64, _i32, _i32, _p, _p, _p, _p, _sz, _p]
_lib.spardl_team_residual_collect.argtypes = [_p, _i64, _i32, _i32, _i64, _i32, _p, _p, _p, _p, _p, _p]
_lib.spardl_bsag_workspace_bytes.argtypes = [_i32, _i32, _i64, _i32]
_lib.spardl_bsag_workspace_bytes.restype = _sz
_lib.spardl_bsag_workspace_init.argtypes = [_i32, _i32, _i64, _i32, _p, _sz, _p]
_lib.spardl_bsag_exchange.argtypes = [_p, _p, _i32, _i32, _i64, _i32, _p, _p, _p, _p, _p, _sz, _p]
_lib.spardl_bsag_residual.argtypes = [_p, _i64, _i32, _i32, _i64, _i32, _p, _p, _p, _p, _p]
for _f in ("residual_add", "residual_add_collect", "residual_collect_index", "block_topk", "sparse_merge_topk", "sparse_merge_topk_noalloc", "allgather_densify", "residual_collect",
           "lazy_topk", "lazy_receive", "lazy_residual_collect", "rsag_workspace_init", "rsag_merge_topk",
           "rsag_residual", "bsag_workspace_init", "bsag_exchange", "bsag_residual", "team_workspace_init",
           "team_residual_add", "team_block_topk", "team_merge_topk", "team_residual_collect"):
    getattr(_lib, "spardl_" + _f).restype = ctypes.c_int


class SpardlError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"spardl_{fn}: {_lib.spardl_strerror(status).decode()} ({status})")
        self.status = status


def _check(fn: str, status: int) -> None:
    if status != OK:
        raise SpardlError(fn, status)


def _ptr(t) -> int:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ld(t, n) -> int:
    return t.stride(0) if t.dim() == 2 else n


def strerror(status: int) -> str:
    return _lib.spardl_strerror(status).decode()


def srs_plan(P: int):
    """(l, distances, bag_blocks) of the Spar-Reduce-Scatter steps."""
    dist = (ctypes.c_int32 * 32)()
    bags = (ctypes.c_int32 * 32)()
    l = _lib.spardl_srs_plan(P, dist, bags)
    if l < 0:
        raise SpardlError("srs_plan", l)
    return l, list(dist[:l]), list(bags[:l])


def workspace_bytes(nworkers: int, P: int, n: int, k_blk: int) -> int:
    return int(_lib.spardl_workspace_bytes(nworkers, P, n, k_blk))


def workspace_init(ws, nworkers: int, P: int, n: int, k_blk: int, *, stream=None) -> None:
    _check("workspace_init", _lib.spardl_workspace_init(nworkers, P, n, k_blk, _ptr(ws),
                                                        ws.numel() * ws.element_size(), _stream(stream)))


def workspace(nworkers: int, P: int, n: int, k_blk: int, device="cuda", *, stream=None):
    """A prepared workspace (uint8 device tensor) for calls with these sizes."""
    ws = torch.empty(workspace_bytes(nworkers, P, n, k_blk), dtype=torch.uint8, device=device)
    workspace_init(ws, nworkers, P, n, k_blk, stream=stream)
    return ws


def residual_add(acc, grad, nworkers: int, n: int, P: int = 0, ws=None, k_blk: int = 0, *, w0: int = 0,
                 ld_acc=None, ld_grad=None, stream=None) -> None:
    """w0: the worker of row 0 when the call covers workers w0 .. w0 + nworkers - 1."""
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    ld_grad = _ld(grad, n) if ld_grad is None else ld_grad
    ws_bytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check("residual_add", _lib.spardl_residual_add(_ptr(acc), ld_acc, _ptr(grad), ld_grad, w0, nworkers, n, P,
                                                    k_blk, _ptr(ws), ws_bytes, _stream(stream)))


def residual_add_collect(acc, grad, nworkers: int, n: int, P: int, ws, k_blk: int, local_idx, member, drop_idx,
                         drop_val, drop_cnt, *, w0: int = 0, ld_acc=None, ld_grad=None, stream=None) -> None:
    """The previous step's residual collection fused into this step's add.
    acc / grad / local_idx: the rows w0 .. w0 + nworkers - 1; member and
    drop_* (sequences of l tensors, one per SRS step) as for residual_collect."""
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    ld_grad = _ld(grad, n) if ld_grad is None else ld_grad
    l = len(drop_idx)
    arr = lambda ts: (ctypes.c_void_p * max(l, 1))(*[_ptr(t) for t in ts]) if l else None
    _check("residual_add_collect", _lib.spardl_residual_add_collect(
        _ptr(acc), ld_acc, _ptr(grad), ld_grad, w0, nworkers, n, P, k_blk, _ptr(local_idx), _ptr(member),
        arr(drop_idx), arr(drop_val), arr(drop_cnt), _ptr(ws), _nb(ws), _stream(stream)))


def residual_collect_index(w0: int, nworkers: int, n: int, P: int, k_blk: int, drop_idx, drop_cnt, ws, *,
                           stream=None) -> None:
    """The drop-tile index the next residual_add_collect of rows w0 .. w0 + nworkers - 1 reads."""
    l = len(drop_idx)
    arr = lambda ts: (ctypes.c_void_p * max(l, 1))(*[_ptr(t) for t in ts]) if l else None
    _check("residual_collect_index", _lib.spardl_residual_collect_index(
        w0, nworkers, n, P, k_blk, arr(drop_idx), arr(drop_cnt), _ptr(ws), _nb(ws), _stream(stream)))


def block_topk(acc, nworkers: int, n: int, P: int, k_blk: int, sp_idx, sp_val, local_idx=None, ws=None,
               flags: int = 0, *, w0: int = 0, ld_acc=None, stream=None) -> None:
    """w0: the worker of row 0 when the call covers workers w0 .. w0 + nworkers - 1."""
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    _check("block_topk", _lib.spardl_block_topk(_ptr(acc), ld_acc, w0, nworkers, n, P, k_blk, flags, _ptr(sp_idx),
                                                _ptr(sp_val), _ptr(local_idx), _ptr(ws),
                                                ws.numel() * ws.element_size(), _stream(stream)))


def sparse_merge_topk(sp_idx, sp_val, P: int, n: int, k_blk: int, round: int, drop_idx, drop_val, drop_cnt,
                      ws, *, stream=None) -> None:
    _check("sparse_merge_topk", _lib.spardl_sparse_merge_topk(
        _ptr(sp_idx), _ptr(sp_val), P, n, k_blk, round, _ptr(drop_idx), _ptr(drop_val), _ptr(drop_cnt),
        _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 64 << 20


def sparse_merge_topk_noalloc(sp_idx, sp_val, P: int, n: int, k_blk: int, round: int, drop_idx, drop_val,
                              drop_cnt, err, *, stream=None) -> None:
    """The SRS step without a workspace (the library's static scratch); err: a
    4-byte device tensor the call clears and its kernels OR error bits into."""
    _check("sparse_merge_topk_noalloc", _lib.spardl_sparse_merge_topk_noalloc(
        _ptr(sp_idx), _ptr(sp_val), P, n, k_blk, round, _ptr(drop_idx), _ptr(drop_val), _ptr(drop_cnt), _ptr(err),
        _stream(stream)))


def member_words(n: int) -> int:
    """Words of the membership bitmap of the final index set."""
    return (n + 31) // 32


def allgather_densify(sp_idx, sp_val, P: int, n: int, k_blk: int, dense, member=None, *, stream=None) -> None:
    """member: optional int32 tensor of member_words(n) words, receives the bitmap of I."""
    _check("allgather_densify", _lib.spardl_allgather_densify(_ptr(sp_idx), _ptr(sp_val), P, n, k_blk,
                                                              _ptr(dense), _ptr(member), _stream(stream)))


def residual_collect(acc, P: int, n: int, k_blk: int, local_idx, sp_idx, drop_idx, drop_val, drop_cnt, ws,
                     member=None, *, ld_acc=None, stream=None) -> None:
    """drop_idx / drop_val / drop_cnt: sequences of l tensors (one per step).
    member: the bitmap allgather_densify wrote (then sp_idx and ws may be None)."""
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    l = len(drop_idx)
    arr = lambda ts: (ctypes.c_void_p * max(l, 1))(*[_ptr(t) for t in ts]) if l else None
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("residual_collect", _lib.spardl_residual_collect(
        _ptr(acc), ld_acc, P, n, k_blk, _ptr(local_idx), _ptr(sp_idx), _ptr(member), arr(drop_idx),
        arr(drop_val), arr(drop_cnt), _ptr(ws), ws_bytes, _stream(stream)))


def lazy_topk(acc, w0: int, nworkers: int, n: int, P: int, k_blk: int, round: int, sp_idx, sp_val, ws,
              flags: int = 0, *, ld_acc=None, stream=None) -> None:
    """acc: rows w0 .. w0 + nworkers - 1; sp_idx/sp_val: sp[w0:w0 + nworkers]."""
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    _check("lazy_topk", _lib.spardl_lazy_topk(_ptr(acc), ld_acc, w0, nworkers, n, P, k_blk, round, flags,
                                              _ptr(sp_idx), _ptr(sp_val), _ptr(ws), ws.numel() * ws.element_size(),
                                              _stream(stream)))


def lazy_receive(acc, P: int, n: int, k_blk: int, round: int, sp_idx, sp_val, saved, ws=None, *, ld_acc=None,
                 stream=None) -> None:
    """ws: the fused form's workspace (keeps the add's histograms exact), or None."""
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("lazy_receive", _lib.spardl_lazy_receive(_ptr(acc), ld_acc, P, n, k_blk, round, _ptr(sp_idx),
                                                    _ptr(sp_val), _ptr(saved), _ptr(ws), ws_bytes,
                                                    _stream(stream)))


def lazy_residual_collect(acc, P: int, n: int, k_blk: int, sp_idx, member, saved, *, ld_acc=None,
                          stream=None) -> None:
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    _check("lazy_residual_collect", _lib.spardl_lazy_residual_collect(
        _ptr(acc), ld_acc, P, n, k_blk, _ptr(sp_idx), _ptr(member), _ptr(saved), _stream(stream)))


def rsag_workspace(P: int, d: int, n: int, k_blk: int, device="cuda", *, stream=None):
    """A prepared workspace for spardl_rsag_merge_topk with these sizes."""
    nbytes = int(_lib.spardl_rsag_workspace_bytes(P, d, n, k_blk))
    if nbytes == 0:
        raise SpardlError("rsag_workspace_bytes", EINVAL)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    _check("rsag_workspace_init", _lib.spardl_rsag_workspace_init(P, d, n, k_blk, _ptr(ws), nbytes, _stream(stream)))
    return ws


def rsag_merge_topk(sp_idx, sp_val, P: int, d: int, n: int, k_blk: int, t: int, drop_idx, drop_val, drop_cnt, ws,
                    *, stream=None) -> None:
    _check("rsag_merge_topk", _lib.spardl_rsag_merge_topk(
        _ptr(sp_idx), _ptr(sp_val), P, d, n, k_blk, t, _ptr(drop_idx), _ptr(drop_val), _ptr(drop_cnt), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def rsag_residual(acc, P: int, d: int, n: int, k_blk: int, member, drop_idx, drop_val, drop_cnt, *, ld_acc=None,
                  stream=None) -> None:
    """drop_*: sequences of log2(d) tensors (one per exchange)."""
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    steps = len(drop_idx)
    arr = lambda ts: (ctypes.c_void_p * max(steps, 1))(*[_ptr(t) for t in ts])
    _check("rsag_residual", _lib.spardl_rsag_residual(_ptr(acc), ld_acc, P, d, n, k_blk, _ptr(member),
                                                      arr(drop_idx), arr(drop_val), arr(drop_cnt),
                                                      _stream(stream)))


def team_workspace(P: int, d: int, n: int, k_blk: int, device="cuda", *, stream=None):
    """A prepared workspace for the team calls (all d teams at once)."""
    nbytes = int(_lib.spardl_team_workspace_bytes(P, d, n, k_blk))
    if nbytes == 0:
        raise SpardlError("team_workspace_bytes", EINVAL)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    _check("team_workspace_init", _lib.spardl_team_workspace_init(P, d, n, k_blk, _ptr(ws), nbytes, _stream(stream)))
    return ws


def _nb(ws) -> int:
    return ws.numel() * ws.element_size()


def team_residual_add(acc, grad, P: int, d: int, n: int, k_blk: int, ws, *, stream=None) -> None:
    _check("team_residual_add", _lib.spardl_team_residual_add(_ptr(acc), _ld(acc, n), _ptr(grad), _ld(grad, n), P, d,
                                                              n, k_blk, _ptr(ws), _nb(ws), _stream(stream)))


def team_block_topk(acc, P: int, d: int, n: int, k_blk: int, sp_idx, sp_val, local_idx, ws, flags: int = 0, *,
                    stream=None) -> None:
    _check("team_block_topk", _lib.spardl_team_block_topk(_ptr(acc), _ld(acc, n), P, d, n, k_blk, flags,
                                                          _ptr(sp_idx), _ptr(sp_val), _ptr(local_idx), _ptr(ws),
                                                          _nb(ws), _stream(stream)))


def team_merge_topk(sp_idx, sp_val, P: int, d: int, n: int, k_blk: int, round: int, drop_idx, drop_val, drop_cnt,
                    ws, *, stream=None) -> None:
    _check("team_merge_topk", _lib.spardl_team_merge_topk(_ptr(sp_idx), _ptr(sp_val), P, d, n, k_blk, round,
                                                          _ptr(drop_idx), _ptr(drop_val), _ptr(drop_cnt), _ptr(ws),
                                                          _nb(ws), _stream(stream)))


def team_residual_collect(acc, P: int, d: int, n: int, k_blk: int, local_idx, member, drop_idx, drop_val, drop_cnt,
                          *, ld_acc=None, stream=None) -> None:
    """drop_*: sequences of ceil(log2(P / d)) tensors (the team_merge_topk buffers, one per round)."""
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    l = len(drop_idx)
    arr = lambda ts: (ctypes.c_void_p * max(l, 1))(*[_ptr(t) for t in ts]) if l else None
    _check("team_residual_collect", _lib.spardl_team_residual_collect(
        _ptr(acc), ld_acc, P, d, n, k_blk, _ptr(local_idx), _ptr(member), arr(drop_idx), arr(drop_val),
        arr(drop_cnt), _stream(stream)))


def bsag_workspace(P: int, d: int, n: int, k_blk: int, device="cuda", *, stream=None):
    """A prepared workspace for spardl_bsag_exchange (it carries Algorithm 2's state)."""
    nbytes = int(_lib.spardl_bsag_workspace_bytes(P, d, n, k_blk))
    if nbytes == 0:
        raise SpardlError("bsag_workspace_bytes", EINVAL)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    _check("bsag_workspace_init", _lib.spardl_bsag_workspace_init(P, d, n, k_blk, _ptr(ws), nbytes, _stream(stream)))
    return ws


def bsag_exchange(sp_idx, sp_val, P: int, d: int, n: int, k_blk: int, drop_idx, drop_val, drop_cnt, ws, info=None,
                  *, stream=None) -> None:
    _check("bsag_exchange", _lib.spardl_bsag_exchange(
        _ptr(sp_idx), _ptr(sp_val), P, d, n, k_blk, _ptr(drop_idx), _ptr(drop_val), _ptr(drop_cnt), _ptr(info),
        _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def bsag_residual(acc, P: int, d: int, n: int, k_blk: int, member, drop_idx, drop_val, drop_cnt, *, ld_acc=None,
                  stream=None) -> None:
    ld_acc = _ld(acc, n) if ld_acc is None else ld_acc
    _check("bsag_residual", _lib.spardl_bsag_residual(_ptr(acc), ld_acc, P, d, n, k_blk, _ptr(member),
                                                      _ptr(drop_idx), _ptr(drop_val), _ptr(drop_cnt),
                                                      _stream(stream)))


def ws_layout(P: int, n: int, kb: int, ws_bytes: int) -> dict:
    """Byte offsets of the arrays in a workspace of spardl_workspace_bytes(...,
    P, n, kb) (host bookkeeping mirroring csrc/api.hip's layout, for reading
    per-block statistics; tests/test_abi_cpu.py keeps the two in step)."""
    al = lambda x: (x + 255) & ~255
    l = 0
    while (1 << l) < P:
        l += 1
    bags = [P - (1 << (l - 1)) if i == 1 else (1 << (l - i)) for i in range(1, l + 1)]
    mmax = max(bags) if bags else 0
    maxlen = -(-n // P)
    pairs_max = P * mmax
    units = max(P * P, pairs_max)
    tiles_tk = -(-(maxlen + 31) // 4096)     # slots and add tiles start at a block's 32-aligned origin
    tiles_mg = -(-2 * kb // 4096)
    add_tiles = -(-(maxlen + 31) // 2048)
    slot_n = max(P * P * tiles_tk, pairs_max * tiles_mg)
    L, off = {"add_tiles": add_tiles}, 256
    L["bitmap"] = off; off += al(-(-n // 32) * 4)
    copies = 4                                           # level-1 histogram copies per unit: one per ~512
    while copies < 32 and copies * 512 < add_tiles:      # add tiles of a block, a power of two in [4, 32]
        copies *= 2
    L["hcopies"] = copies
    L["hist1"] = off; off += al(units * copies * 4096 * 4)
    L["spec_t1"] = off; off += al(P * P * 4)
    L["spec_used"] = off; off += al(P * P * 4)
    L["spec_cnt"] = off; off += al(P * P * add_tiles * 4)
    L["state"] = off; off += al(units * 16 * 4)
    for k in ("slot_cnt", "slot_nbin", "pre_all", "pre_ge", "pre_eq"):
        L[k] = off; off += al(slot_n * 4)
    L["keep"] = off; off += al(P * P * 4 * 4)             # the block top-k's selection rule per (worker, block)
    L["dtile"] = off; off += al(sum(P * m for m in bags) * add_tiles * 8)   # per (step, pair, add tile)
    L["fixed_end"] = off
    L["cand_entries"] = max(P * n, pairs_max * tiles_mg * 4096)
    q = ((ws_bytes - off) // 3) & ~255
    L["cand_idx"], L["cand_val"], L["bin_key"] = off, off + q, off + 2 * q
    return L


def topk_stats(ws, rows: int, P: int, n: int, kb: int) -> dict:
    """After spardl_residual_add (fused) and spardl_block_topk on `rows` rows:
    per (row, block), the speculative candidates the add wrote and whether the
    selection used them instead of reading the block again (reads the
    workspace; synchronises the current stream)."""
    L = ws_layout(P, n, kb, ws.numel())
    G = L["add_tiles"]
    cnt = ws[L["spec_cnt"]:L["spec_cnt"] + rows * P * G * 4].view(torch.int32).cpu().view(rows * P, G)
    state = ws[L["state"]:L["state"] + rows * P * 16 * 4].view(torch.int32).cpu().view(rows * P, 16)
    cands, used = [], []
    for u in range(rows * P):
        b = u % P
        s, e = (b * n) // P, ((b + 1) * n) // P
        tiles = -(-(e - s + (s & 31)) // 2048)   # the block's tiles (the rest of the row's slots are unused)
        cands.append(int(cnt[u, :tiles].clamp(min=0).sum()))
        used.append(bool(state[u, 7]))
    return {"candidates": cands, "spec_ok": used}


def ws_error(ws) -> int:
    """Error word at the start of a workspace (synchronises the current stream)."""
    return int(ws[:4].view(torch.int32).cpu().item())


class _Checkpoint:
    """What a later step needs from the earlier ones (Algorithm 1's input
    residual xi^{t-1}; for B-SAG also Algorithm 2's per-block h, step, flag
    and N, which live in its workspace), copied to host memory and back.
    Everything else a step object holds is recomputed by the next step; a
    fresh object's speculation hints are empty, which only makes its first
    top-k read the blocks once more."""

    def state_dict(self) -> dict:
        d = {"acc": self.acc.cpu()}
        if getattr(self, "bruck", False):
            d["bsag_ws"] = self.ws_sag.cpu()
        return d

    def load_state_dict(self, d: dict) -> None:
        self.acc.copy_(d["acc"])
        if getattr(self, "bruck", False):
            self.ws_sag.copy_(d["bsag_ws"])


class SparDLStep(_Checkpoint):
    """Buffers for P simulated workers and one synchronisation step through the C ABI.

    acc[P, n] holds the residual between steps.  After step(grad): dense holds
    the global update, sp_idx/sp_val the sparse state (final block b in
    sp[b, b]), local_idx the local selections and drop_* the per-step drops.
    With fuse_collect, a step leaves its residual collection to the next
    step's add (spardl_residual_add_collect): acc holds the residual only
    after flush(), which runs the pending collection on its own.
    """

    def __init__(self, P: int, n: int, k_blk: int, device="cuda", fused: bool = True, rows_per_call: int = 0,
                 fuse_collect: bool = False):
        """rows_per_call: workers per residual-add / block top-k call (0: all P).
        The workspace is sized for that many rows, so a model too large for a
        P-row workspace runs its workers a few at a time."""
        if fuse_collect and not fused:
            raise ValueError("the collection fuses into the fused residual add only")
        self.P, self.n, self.k_blk, self.fused = P, n, k_blk, fused
        self.fuse_collect = fuse_collect
        self.pending = [False] * P   # per worker: its residual collection waits for its next add
        self.rows = P if rows_per_call <= 0 else min(rows_per_call, P)
        dev = torch.device(device)
        self.acc = torch.zeros((P, n), dtype=torch.float32, device=dev)
        self.sp_idx = torch.empty((P, P, k_blk), dtype=torch.int32, device=dev)
        self.sp_val = torch.empty((P, P, k_blk), dtype=torch.float32, device=dev)
        self.local_idx = torch.empty((P, P, k_blk), dtype=torch.int32, device=dev)
        self.l, self.distance, self.bags = srs_plan(P)
        self.drop_idx = [torch.empty((P, m, k_blk), dtype=torch.int32, device=dev) for m in self.bags]
        self.drop_val = [torch.empty((P, m, k_blk), dtype=torch.float32, device=dev) for m in self.bags]
        self.drop_cnt = [torch.empty((P, m), dtype=torch.int32, device=dev) for m in self.bags]
        self.dense = torch.empty(n, dtype=torch.float32, device=dev)
        self.member = torch.empty(member_words(n), dtype=torch.int32, device=dev)
        self.ws = workspace(self.rows, P, n, k_blk, device=dev)

    def residual_add_rows(self, w0: int, grad_rows, stream=None):
        """Rows w0 .. w0 + len(grad_rows) - 1 (at most rows_per_call)."""
        r = grad_rows.shape[0]
        acc = self.acc[w0:w0 + r]
        pend = self.pending[w0:w0 + r]
        if any(pend) and not all(pend):
            raise ValueError("rows with and without a pending collection in one call")
        if pend and pend[0]:
            residual_add_collect(acc, grad_rows, r, self.n, self.P, self.ws, self.k_blk, self.local_idx[w0:w0 + r],
                                 self.member, self.drop_idx, self.drop_val, self.drop_cnt, w0=w0, stream=stream)
            self.pending[w0:w0 + r] = [False] * r
        elif self.fused:
            residual_add(acc, grad_rows, r, self.n, self.P, self.ws, self.k_blk, w0=w0, stream=stream)
        else:
            residual_add(acc, grad_rows, r, self.n, 0, None, stream=stream)

    def block_topk_rows(self, w0: int, r: int, stream=None):
        s = slice(w0, w0 + r)
        block_topk(self.acc[s], r, self.n, self.P, self.k_blk, self.sp_idx[s], self.sp_val[s], self.local_idx[s],
                   self.ws, TOPK_HIST_READY if self.fused else 0, w0=w0, stream=stream)

    def residual_add(self, grad, stream=None):
        self._all_rows()
        self.residual_add_rows(0, grad, stream)

    def block_topk(self, stream=None):
        self._all_rows()
        self.block_topk_rows(0, self.P, stream)

    def _all_rows(self):
        if self.rows != self.P:
            raise ValueError("a workspace for fewer rows than P: alternate residual_add_rows and "
                             "block_topk_rows per worker group (step() does)")

    def merge_round(self, i: int, stream=None):
        sparse_merge_topk(self.sp_idx, self.sp_val, self.P, self.n, self.k_blk, i, self.drop_idx[i - 1],
                          self.drop_val[i - 1], self.drop_cnt[i - 1], self.ws, stream=stream)

    def densify(self, stream=None):
        allgather_densify(self.sp_idx, self.sp_val, self.P, self.n, self.k_blk, self.dense,
                          self.member if self.fused else None, stream=stream)

    def collect(self, stream=None):
        """The residual collection now (with fuse_collect: the next add's, after
        which acc holds the residual)."""
        if self.fuse_collect:
            residual_collect_index(0, self.P, self.n, self.P, self.k_blk, self.drop_idx, self.drop_cnt, self.ws,
                                   stream=stream)
            self.pending = [True] * self.P
            return
        self._collect(stream)

    def _collect(self, stream=None):
        residual_collect(self.acc, self.P, self.n, self.k_blk, self.local_idx, self.sp_idx, self.drop_idx,
                         self.drop_val, self.drop_cnt, self.ws, self.member if self.fused else None,
                         stream=stream)

    def flush(self, stream=None):
        """Run a pending residual collection on its own, so that acc holds the residual
        (the drop-tile index built for it is cleared by the next index build's
        consumer, so a fresh workspace state is restored here)."""
        if any(self.pending):
            if not all(self.pending):
                raise ValueError("a partly applied collection")
            self._collect(stream)
            self.pending = [False] * self.P

    def state_dict(self) -> dict:
        self.flush()
        return super().state_dict()

    def load_state_dict(self, d: dict) -> None:
        super().load_state_dict(d)
        self.pending = [False] * self.P

    def finish(self, stream=None):
        """The SRS steps, the decode and the residual collection, after every
        worker's residual add and block top-k."""
        for i in range(1, self.l + 1):
            self.merge_round(i, stream)
        self.densify(stream)
        self.collect(stream)

    def step(self, grad, stream=None):
        if self.rows == self.P:
            self.residual_add(grad, stream)
            self.block_topk(stream)
        else:   # a worker group's add and top-k share the workspace, so they alternate
            for w0 in range(0, self.P, self.rows):
                r = min(self.rows, self.P - w0)
                self.residual_add_rows(w0, grad[w0:w0 + r], stream)
                self.block_topk_rows(w0, r, stream)
        self.finish(stream)


class SparDLLazyStep(_Checkpoint):
    """Buffers for P simulated workers and one lazy-sparsification step
    (Sec. III-B "Optimization for SRS", Algorithm 1) through the C ABI.

    acc[P, n] holds the residual between steps (and the workers' dense blocks
    during a step).  After step(grad): dense holds the global update, member
    the bitmap of its index set, sp_idx/sp_val[w, b] worker w's selection of
    block b (final block b in sp[b, b]), saved what the receipts overwrote.
    """

    def __init__(self, P: int, n: int, k_blk: int, device="cuda", rows_per_call: int = 0, fused: bool = True):
        """fused: the add prepares every block's selection and the receipts keep
        it exact (needs all P rows in one workspace, so rows_per_call < P
        runs the plain form)."""
        self.P, self.n, self.k_blk = P, n, k_blk
        self.rows = P if rows_per_call <= 0 else min(rows_per_call, P)
        self.fused = fused and self.rows == P
        dev = torch.device(device)
        self.acc = torch.zeros((P, n), dtype=torch.float32, device=dev)
        self.sp_idx = torch.empty((P, P, k_blk), dtype=torch.int32, device=dev)
        self.sp_val = torch.empty((P, P, k_blk), dtype=torch.float32, device=dev)
        self.saved = torch.empty((P, P, k_blk), dtype=torch.float32, device=dev)
        self.l, self.distance, self.bags = srs_plan(P)
        self.dense = torch.empty(n, dtype=torch.float32, device=dev)
        self.member = torch.empty(member_words(n), dtype=torch.int32, device=dev)
        self.ws = workspace(self.rows, P, n, k_blk, device=dev)

    def residual_add_rows(self, w0: int, grad_rows, stream=None):
        r = grad_rows.shape[0]
        if self.fused:
            if w0 != 0 or r != self.P:
                raise ValueError("the fused lazy step adds all P rows in one call")
            residual_add(self.acc, grad_rows, r, self.n, self.P, self.ws, self.k_blk, stream=stream)
        else:
            residual_add(self.acc[w0:w0 + r], grad_rows, r, self.n, 0, None, stream=stream)

    def topk_round(self, i: int, stream=None):
        """Every worker's selection for step i (0: the reserved blocks)."""
        flags = TOPK_HIST_READY if self.fused else 0
        for w0 in range(0, self.P, self.rows):
            r = min(self.rows, self.P - w0)
            s = slice(w0, w0 + r)
            lazy_topk(self.acc[s], w0, r, self.n, self.P, self.k_blk, i, self.sp_idx[s], self.sp_val[s], self.ws,
                      flags, stream=stream)

    def receive(self, i: int, stream=None):
        lazy_receive(self.acc, self.P, self.n, self.k_blk, i, self.sp_idx, self.sp_val, self.saved,
                     self.ws if self.fused else None, stream=stream)

    def densify(self, stream=None):
        allgather_densify(self.sp_idx, self.sp_val, self.P, self.n, self.k_blk, self.dense, self.member,
                          stream=stream)

    def collect(self, stream=None):
        lazy_residual_collect(self.acc, self.P, self.n, self.k_blk, self.sp_idx, self.member,
                              self.saved if self.l else None, stream=stream)

    def finish(self, stream=None):
        """Everything after the residual add of every worker."""
        for i in range(1, self.l + 1):
            self.topk_round(i, stream)
            self.receive(i, stream)
        self.topk_round(0, stream)
        self.densify(stream)
        self.collect(stream)

    def step(self, grad, stream=None):
        self.residual_add_rows(0, grad, stream)
        self.finish(stream)


class SparDLSagStep(_Checkpoint):
    """P simulated workers in d teams of Q = P / d joined by R-SAG (Sec. III-D,
    d a power of 2) or, with bruck=True, by B-SAG (any d dividing P, top-h
    counts from Algorithm 2), one synchronisation step through the C ABI.

    k_blk is L(k, d, P) = d k / P, the entries per block of a team's Q blocks.
    After step(grad): dense / member as for SparDLStep; sp_idx/sp_val[w, b]
    the state of worker w's block b (final block q in sp[q, q] of every
    team); drop_*[i - 1][w] the SRS drops of worker w at step i inside its
    team; sag_*[t][p] what pair p dropped at exchange t.
    """

    def __init__(self, P: int, d: int, n: int, k_blk: int, device="cuda", fused: bool = True, bruck: bool = False,
                 batched: bool = True):
        """batched: the teams' add, top-k and SRS steps in one call each over
        all P rows (otherwise team by team, each with its own workspace)."""
        if d < 2 or P % d or (not bruck and d & (d - 1)):
            raise ValueError("d >= 2 must divide P (and be a power of two for R-SAG)")
        self.P, self.d, self.Q, self.n, self.k_blk, self.fused = P, d, P // d, n, k_blk, fused
        self.bruck, self.batched = bruck, batched
        Q = self.Q
        dev = torch.device(device)
        self.acc = torch.zeros((P, n), dtype=torch.float32, device=dev)
        self.sp_idx = torch.empty((P, Q, k_blk), dtype=torch.int32, device=dev)
        self.sp_val = torch.empty((P, Q, k_blk), dtype=torch.float32, device=dev)
        self.local_idx = torch.empty((P, Q, k_blk), dtype=torch.int32, device=dev)
        self.l, self.distance, self.bags = srs_plan(Q)
        self.drop_idx = [torch.empty((P, m, k_blk), dtype=torch.int32, device=dev) for m in self.bags]
        self.drop_val = [torch.empty((P, m, k_blk), dtype=torch.float32, device=dev) for m in self.bags]
        self.drop_cnt = [torch.empty((P, m), dtype=torch.int32, device=dev) for m in self.bags]
        self.dense = torch.empty(n, dtype=torch.float32, device=dev)
        self.member = torch.empty(member_words(n), dtype=torch.int32, device=dev)
        if batched:
            self.ws_all = team_workspace(P, d, n, k_blk, device=dev)
            self.ws_team = [self.ws_all]    # (its error word is checked like the per-team ones)
        else:
            self.ws_team = [workspace(Q, Q, n, k_blk, device=dev) for _ in range(d)]
        if bruck:
            self.steps = 1
            self.toph_idx = torch.empty((P, k_blk), dtype=torch.int32, device=dev)
            self.toph_val = torch.empty((P, k_blk), dtype=torch.float32, device=dev)
            self.toph_cnt = torch.empty(P, dtype=torch.int32, device=dev)
            self.info = torch.empty(2 * Q, dtype=torch.int32, device=dev)
            self.ws_sag = bsag_workspace(P, d, n, k_blk, device=dev)
        else:
            self.steps = d.bit_length() - 1
            npairs = (d // 2) * Q
            self.sag_idx = [torch.empty((npairs, k_blk), dtype=torch.int32, device=dev) for _ in range(self.steps)]
            self.sag_val = [torch.empty((npairs, k_blk), dtype=torch.float32, device=dev) for _ in range(self.steps)]
            self.sag_cnt = [torch.empty(npairs, dtype=torch.int32, device=dev) for _ in range(self.steps)]
            self.ws_sag = rsag_workspace(P, d, n, k_blk, device=dev)

    def _rows(self, tau):
        return slice(tau * self.Q, (tau + 1) * self.Q)

    def add_and_select(self, grad, stream=None):
        Q, n, L = self.Q, self.n, self.k_blk
        if self.batched:
            if self.fused:
                team_residual_add(self.acc, grad, self.P, self.d, n, L, self.ws_all, stream=stream)
            else:
                residual_add(self.acc, grad, self.P, n, 0, None, stream=stream)
            team_block_topk(self.acc, self.P, self.d, n, L, self.sp_idx, self.sp_val, self.local_idx, self.ws_all,
                            TOPK_HIST_READY if self.fused else 0, stream=stream)
            return
        for tau in range(self.d):
            r, ws = self._rows(tau), self.ws_team[tau]
            if self.fused:
                residual_add(self.acc[r], grad[r], Q, n, Q, ws, L, stream=stream)
            else:
                residual_add(self.acc[r], grad[r], Q, n, 0, None, stream=stream)
            block_topk(self.acc[r], Q, n, Q, L, self.sp_idx[r], self.sp_val[r], self.local_idx[r], ws,
                       TOPK_HIST_READY if self.fused else 0, stream=stream)

    def team_srs(self, stream=None):
        if self.batched:
            for i in range(1, self.l + 1):
                team_merge_topk(self.sp_idx, self.sp_val, self.P, self.d, self.n, self.k_blk, i, self.drop_idx[i - 1],
                                self.drop_val[i - 1], self.drop_cnt[i - 1], self.ws_all, stream=stream)
            return
        for tau in range(self.d):
            r = self._rows(tau)
            for i in range(1, self.l + 1):
                sparse_merge_topk(self.sp_idx[r], self.sp_val[r], self.Q, self.n, self.k_blk, i,
                                  self.drop_idx[i - 1][r], self.drop_val[i - 1][r], self.drop_cnt[i - 1][r],
                                  self.ws_team[tau], stream=stream)

    def exchanges(self, stream=None):
        if self.bruck:
            bsag_exchange(self.sp_idx, self.sp_val, self.P, self.d, self.n, self.k_blk, self.toph_idx,
                          self.toph_val, self.toph_cnt, self.ws_sag, self.info, stream=stream)
            return
        for t in range(self.steps):
            rsag_merge_topk(self.sp_idx, self.sp_val, self.P, self.d, self.n, self.k_blk, t, self.sag_idx[t],
                            self.sag_val[t], self.sag_cnt[t], self.ws_sag, stream=stream)

    def densify(self, stream=None):
        Q = self.Q
        allgather_densify(self.sp_idx[:Q], self.sp_val[:Q], Q, self.n, self.k_blk, self.dense, self.member,
                          stream=stream)

    def collect(self, stream=None):
        if self.batched:
            team_residual_collect(self.acc, self.P, self.d, self.n, self.k_blk, self.local_idx, self.member,
                                  self.drop_idx, self.drop_val, self.drop_cnt, stream=stream)
        else:
            for tau in range(self.d):
                r = self._rows(tau)
                residual_collect(self.acc[r], self.Q, self.n, self.k_blk, self.local_idx[r], self.sp_idx[r],
                                 [t[r] for t in self.drop_idx], [t[r] for t in self.drop_val],
                                 [t[r] for t in self.drop_cnt], None, self.member, stream=stream)
        if self.bruck:
            bsag_residual(self.acc, self.P, self.d, self.n, self.k_blk, self.member, self.toph_idx, self.toph_val,
                          self.toph_cnt, stream=stream)
        else:
            rsag_residual(self.acc, self.P, self.d, self.n, self.k_blk, self.member, self.sag_idx, self.sag_val,
                          self.sag_cnt, stream=stream)

    def step(self, grad, stream=None):
        self.add_and_select(grad, stream)
        self.team_srs(stream)
        self.exchanges(stream)
        self.densify(stream)
        self.collect(stream)
