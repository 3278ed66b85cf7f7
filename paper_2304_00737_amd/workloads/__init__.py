"""Seeded synthetic gradient workloads (input plumbing; none of the method's arithmetic).

The paper trains real models (Table 2); their datasets and weights are not
available here, so gradients are synthesised with the sizes and value
structure of those models: contiguous layer segments, a per-segment scale
drawn log-uniformly, and a per-config value distribution.  Every value is a
pure function of (config, step, worker, element), computed by the C generator
in gradgen.h / gradgen.c, so any slice can be regenerated on demand.

The same host arrays feed both the CPU oracle and the GPU path.
"""

from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import numpy as np

SEED_BASE = 230400737
_M64 = (1 << 64) - 1
_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgradgen.so")

DIST_CODE = {"normal": 0, "laplace": 1, "student_t3": 2}


def mix64(z: int) -> int:
    """SplitMix64 finaliser (Steele, Lea, Flood 2014), on Python ints."""
    z &= _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def _uniform(key: int, counter: int) -> float:
    h = mix64(key + (counter + 1) * 0x9E3779B97F4A7C15)
    return ((h >> 11) + 0.5) * 2.0 ** -53


def stream_key(cfg_id: int, step: int, worker: int) -> int:
    """Key of worker `worker`'s gradient at step `step` (1-based) of a config."""
    return mix64(mix64(mix64(SEED_BASE ^ ((cfg_id & 0xFF) << 56)) + step) + worker)


def _loguniform(lo: float, hi: float, u: float) -> float:
    return math.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))


def _largest_remainder(weights, total):
    s = sum(weights)
    raw = [w * total / s for w in weights]
    base = [int(math.floor(r)) for r in raw]
    rest = total - sum(base)
    order = sorted(range(len(raw)), key=lambda i: (-(raw[i] - base[i]), i))
    for i in order[:rest]:
        base[i] += 1
    return base


@dataclass(frozen=True)
class Workload:
    """One synthetic configuration: P workers, n fp32 per worker, density num/den."""

    cfg_id: int
    name: str
    P: int
    n: int
    density: tuple
    steps: int
    dist: str
    seg_len: tuple
    seg_scale: tuple
    zero_prob: float = 0.0

    @property
    def k(self) -> int:
        num, den = self.density
        return (self.n * num + den - 1) // den          # k = ceil(rho n)

    @property
    def k_blk(self) -> int:
        shortest = min(((b + 1) * self.n) // self.P - (b * self.n) // self.P for b in range(self.P))
        return min((self.k + self.P - 1) // self.P, shortest)   # k/P rounded up

    @property
    def seg_start(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seg_len)]).astype(np.int64)

    def describe(self) -> dict:
        return {"workload": self.name, "P": self.P, "n_per_worker": self.n,
                "density": f"{self.density[0]}/{self.density[1]}", "k": self.k,
                "k_per_block": self.k_blk, "steps": self.steps, "dist": self.dist,
                "segments": len(self.seg_len), "zero_prob": self.zero_prob, "seed": SEED_BASE}


def _segments_loguniform(cfg_id, count, total, lo_len, hi_len, lo_sc, hi_sc, fixed=None):
    key = mix64(SEED_BASE + 7919 * cfg_id)
    if fixed is None:
        weights = [_loguniform(lo_len, hi_len, _uniform(key, s)) for s in range(count)]
        lens = _largest_remainder(weights, total)
    else:
        pos, size = fixed
        others = [_loguniform(lo_len, hi_len, _uniform(key, s)) for s in range(count - 1)]
        rest = _largest_remainder(others, total - size)
        lens = rest[:pos] + [size] + rest[pos:]
    skey = mix64(key + 1)
    scales = [_loguniform(lo_sc, hi_sc, _uniform(skey, s)) for s in range(count)]
    assert sum(lens) == total and min(lens) > 0
    return tuple(lens), tuple(scales)


def config(cfg_id: int) -> Workload:
    """The five synthetic workloads (model sizes from the paper's Table 2 cases)."""
    if cfg_id == 1:
        n = 1 << 20
        return Workload(1, "iid-normal P=4 n=2^20 rho=1%", 4, n, (1, 100), 1, "normal", (n,), (1.0,))
    if cfg_id == 2:
        n = 25_600_000
        lens, sc = _segments_loguniform(2, 160, n, 2 ** 9, 2 ** 22, 1e-4, 1e-1)
        return Workload(2, "resnet50-sized P=8 n=25.6M rho=1%", 8, n, (1, 100), 3, "normal", lens, sc)
    if cfg_id == 3:
        n = 138_000_000
        lens, sc = _segments_loguniform(3, 16, n, 2 ** 9, 2 ** 22, 1e-5, 1e-2, fixed=(13, 102_760_448))
        return Workload(3, "vgg16-sized P=8 n=138M rho=0.5%", 8, n, (1, 200), 3, "laplace", lens, sc)
    if cfg_id == 4:
        n = 110_000_000
        lens, sc = _segments_loguniform(4, 200, n, 2 ** 9, 2 ** 22, 1e-4, 1e-1)
        return Workload(4, "bert-base-sized P=16 n=110M rho=1% 20% zeros", 16, n, (1, 100), 2,
                        "student_t3", lens, sc, zero_prob=0.2)
    if cfg_id == 5:
        n = 1_500_000_000
        key = mix64(SEED_BASE + 7919 * 5)
        sc = tuple(_loguniform(1e-5, 1e-2, _uniform(mix64(key + 1), s)) for s in range(48))
        return Workload(5, "gpt2-xl-sized P=32 n=1.5B rho=0.1%", 32, n, (1, 1000), 2, "normal",
                        (31_250_000,) * 48, sc)
    raise ValueError(f"unknown config {cfg_id}")


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        lib.gg_fill.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_uint64,
                                ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                ctypes.c_double]
        lib.gg_fill.restype = None
        lib.gg_mix.argtypes = [ctypes.c_uint64]
        lib.gg_mix.restype = ctypes.c_uint64
        lib.gg_log_host.argtypes = [ctypes.c_double]
        lib.gg_log_host.restype = ctypes.c_double
        _lib = lib
    return _lib


def fill(out: np.ndarray, wl: Workload, step: int, worker: int, x0: int = 0) -> np.ndarray:
    """Write elements [x0, x0 + len(out)) of worker `worker`'s gradient at `step`."""
    assert out.dtype == np.float32 and out.flags["C_CONTIGUOUS"]
    lib = _load()
    starts = np.ascontiguousarray(wl.seg_start, dtype=np.int64)
    scales = np.ascontiguousarray(np.array(wl.seg_scale, dtype=np.float64))
    lib.gg_fill(out.ctypes.data, out.size, x0, stream_key(wl.cfg_id, step, worker),
                DIST_CODE[wl.dist], starts.ctypes.data, scales.ctypes.data, len(wl.seg_len),
                float(wl.zero_prob))
    return out


DEV_LIB_PATH = os.path.join(_HERE, "libgradgen_dev.so")
_dev_lib = None


def _load_dev():
    global _dev_lib
    if _dev_lib is None:
        if not os.path.exists(DEV_LIB_PATH):
            raise ImportError(f"{DEV_LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(DEV_LIB_PATH)
        lib.gg_fill_device.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_uint64,
                                       ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                       ctypes.c_double, ctypes.c_void_p]
        lib.gg_fill_device.restype = ctypes.c_int
        _dev_lib = lib
    return _dev_lib


class DeviceGenerator:
    """The same generator on the GPU: fills device memory with the bits fill()
    gives on the host (input plumbing; torch is imported only here)."""

    def __init__(self, wl: Workload, device="cuda"):
        import torch
        self.wl = wl
        self.starts = torch.tensor(np.asarray(wl.seg_start, dtype=np.int64), device=device)
        self.scales = torch.tensor(np.asarray(wl.seg_scale, dtype=np.float64), device=device)
        self.lib = _load_dev()

    def fill(self, out, step: int, worker: int, x0: int = 0, stream=None) -> None:
        """out: contiguous float32 CUDA tensor; element j <- element x0 + j of the gradient."""
        import torch
        assert out.dtype == torch.float32 and out.is_contiguous() and out.is_cuda
        s = (stream or torch.cuda.current_stream()).cuda_stream
        wl = self.wl
        rc = self.lib.gg_fill_device(out.data_ptr(), out.numel(), x0, stream_key(wl.cfg_id, step, worker),
                                     DIST_CODE[wl.dist], self.starts.data_ptr(), self.scales.data_ptr(),
                                     len(wl.seg_len), float(wl.zero_prob), s)
        if rc != 0:
            raise RuntimeError(f"gg_fill_device failed: {rc}")


def gradient(wl: Workload, step: int, worker: int, x0: int = 0, count: int | None = None) -> np.ndarray:
    count = wl.n - x0 if count is None else count
    return fill(np.empty(count, dtype=np.float32), wl, step, worker, x0)


# ---------------------------------------------------------------- small parity shapes


def small_rows(kind: str, P: int, n: int, seed: int) -> np.ndarray:
    """P x n fp32 rows for small parity cases.

    kinds: "normal" (N(0,1)), "ties" (values in {+-1, +-2, +-4} * 2^-8, 30 %
    exact zeros), "dyadic" (integers in [-64, 64], every partial sum exact),
    "const" (every entry -1.5: one giant tie), "zeros" (all +0.0).
    """
    rng = np.random.default_rng(seed)
    if kind == "normal":
        return rng.standard_normal((P, n), dtype=np.float32)
    if kind == "ties":
        v = rng.choice(np.array([1, -1, 2, -2, 4, -4], dtype=np.float32), size=(P, n))
        v[rng.random((P, n)) < 0.3] = 0.0
        return (v * np.float32(2.0 ** -8)).astype(np.float32)
    if kind == "dyadic":
        return rng.integers(-64, 65, size=(P, n)).astype(np.float32)
    if kind == "const":
        return np.full((P, n), -1.5, dtype=np.float32)
    if kind == "zeros":
        return np.zeros((P, n), dtype=np.float32)
    raise ValueError(kind)
