"""Integer checksums of step outputs for the full-size parity tests (test
plumbing: none of the method's arithmetic).

An output of one step on one block index is a stream of 32-bit words (int32
indices and the bit patterns of float32 values) in a fixed order.  Its
checksum is the stream length and two sums over positions i of the stream,

    sum_i (lo16(x_i) * w_a(i) + hi16(x_i) * w_b(i)) mod M,   M = 2^31 - 1,
    w_c(i) = i * c mod M,

for two fixed pairs of odd constants (a, b).  Every term is below 2^31 and
every product below 2^63 for streams shorter than 2^31 words, so the sums are
exact in int64.  The host computes them with numpy on the oracle's outputs
(tests/golden/full_digests.py writes them), the device with torch integer
ops on the GPU's outputs, so a 6 GB block of residual rows never leaves HBM.
A changed, swapped, missing or extra word changes a sum unless the change
happens to cancel modulo M in both sums at once.

The stream order of every output, for each step form, is defined once below
(host_streams / device_streams side by side).
"""

from __future__ import annotations

import numpy as np

M31 = (1 << 31) - 1
CONSTS = ((0x9E3779B1, 0x85EBCA77), (0xC2B2AE3D, 0x27D4EB2F))
CHUNK = 1 << 24


class HostSum:
    def __init__(self):
        self.n = 0
        self.s = [0, 0]

    def add(self, a) -> None:
        x = np.ascontiguousarray(a)
        assert x.dtype.itemsize == 4, x.dtype
        x = x.reshape(-1).view(np.uint32)
        for j0 in range(0, len(x), CHUNK):
            xs = x[j0:j0 + CHUNK].astype(np.int64)
            i = np.arange(self.n + j0, self.n + j0 + len(xs), dtype=np.int64)
            lo, hi = xs & 0xFFFF, xs >> 16
            for k, (ca, cb) in enumerate(CONSTS):
                self.s[k] += int(((lo * ((i * ca) % M31) + hi * ((i * cb) % M31)) % M31).sum())
        self.n += len(x)

    def value(self) -> list:
        return [self.s[0], self.s[1], self.n]


class DeviceSum:
    def __init__(self, device="cuda"):
        import torch
        self.n = 0
        self.acc = torch.zeros(2, dtype=torch.int64, device=device)   # read once, in value()

    def add(self, t) -> None:
        import torch
        t = t.contiguous().reshape(-1)
        assert t.element_size() == 4, t.dtype
        x32 = t.view(torch.int32)
        for j0 in range(0, x32.numel(), CHUNK):
            xs = x32[j0:j0 + CHUNK].to(torch.int64) & 0xFFFFFFFF
            i = torch.arange(self.n + j0, self.n + j0 + xs.numel(), dtype=torch.int64, device=xs.device)
            lo, hi = xs & 0xFFFF, xs >> 16
            for k, (ca, cb) in enumerate(CONSTS):
                self.acc[k] += ((lo * ((i * ca) % M31) + hi * ((i * cb) % M31)) % M31).sum()
        self.n += x32.numel()

    def value(self) -> list:
        s = self.acc.cpu().tolist()
        return [int(s[0]), int(s[1]), self.n]


def _i32(v) -> np.ndarray:
    return np.asarray(v, dtype=np.int32)


def _f32(v) -> np.ndarray:
    return np.asarray(v, dtype=np.float32)


# ---------------------------------------------------------------- stream orders
# host_streams(form, res, ...) -> {name: [numpy arrays in stream order]}
# device_streams(form, st, ...) -> {name: [torch tensors in stream order]}


def host_streams(form: str, res, P: int, b: int, bags, Q: int = 0, d: int = 1, steps: int = 0, L: int = 0) -> dict:
    out = {}
    if form == "eager":
        out["sp"] = [a for w in range(P) for a in (_i32(res.S[(w, b)][0]), _f32(res.S[(w, b)][1]))]
        out["local"] = [_i32(res.local[(w, b)][0]) for w in range(P)]
        dr = []
        for i, m in enumerate(bags, start=1):
            for w in range(P):
                for t in range(m):
                    if (w + t) % P == b:
                        oi, ov = res.drops[(i, w, b)]
                        dr += [_i32([len(oi)]), _i32(oi), _f32(ov)]
        out["drops"] = dr
    elif form == "lazy":
        out["sel"] = [a for w in range(P) for a in (_i32(res.sel[(w, b)][0]), _f32(res.sel[(w, b)][1]))]
    else:   # rsag / bsag, blocks of a team
        out["local"] = [_i32(res.local[(w, b)][0]) for w in range(P)]
        sp = []
        for w in range(P):
            if form == "bsag" and w == b:
                fi, fv = res.final[b]
                sp += [_i32([len(fi)]), _i32(fi), _f32(fv)]
            else:
                sp += [_i32(res.S[(w, b)][0]), _f32(res.S[(w, b)][1])]
        out["sp"] = sp
        dr = []
        for i, m in enumerate(bags, start=1):
            for w in range(P):
                q = w % Q
                for t in range(m):
                    if (q + t) % Q == b:
                        oi, ov = res.drops[(i, w, b)]
                        dr += [_i32([len(oi)]), _i32(oi), _f32(ov)]
        out["drops"] = dr
        if form == "rsag":
            sd = []
            for t in range(steps):
                for p in range((d // 2) * Q):
                    j, q = divmod(p, Q)
                    if q != b:
                        continue
                    low = j & ((1 << t) - 1)
                    X = ((j >> t) << (t + 1)) | low
                    oi, ov = res.sag_drops[(t, X * Q + q)]
                    sd += [_i32([len(oi)]), _i32(oi), _f32(ov)]
            out["sag_drops"] = sd
        else:
            out["info"] = [_i32([res.h[b], len(res.union[b][0])])]
            th = []
            for tau in range(d):
                w = tau * Q + b
                oi, ov = res.drop_h[w]
                th += [_i32([len(oi)]), _i32(oi), _f32(ov)]
            out["toph_drops"] = th
    out["dense"] = [_f32(res.dense[b])]
    out["residual"] = [_f32(res.residual[(w, b)]) for w in range(P)]
    return out


def device_streams(form: str, st, P: int, b: int, lo: int, hi: int, Q: int = 0, d: int = 1) -> dict:
    import torch
    out = {}
    one = lambda c: torch.tensor([int(c)], dtype=torch.int32, device=st.dense.device)
    if form == "eager":
        out["sp"] = [a for w in range(P) for a in (st.sp_idx[w, b], st.sp_val[w, b])]
        out["local"] = [st.local_idx[w, b] for w in range(P)]
        dr = []
        for i, m in enumerate(st.bags, start=1):
            cnt = st.drop_cnt[i - 1].cpu().numpy()
            for w in range(P):
                for t in range(m):
                    if (w + t) % P == b:
                        c = int(cnt[w, t])
                        dr += [one(c), st.drop_idx[i - 1][w, t, :c], st.drop_val[i - 1][w, t, :c]]
        out["drops"] = dr
    elif form == "lazy":
        out["sel"] = [a for w in range(P) for a in (st.sp_idx[w, b], st.sp_val[w, b])]
    else:
        out["local"] = [st.local_idx[w, b] for w in range(P)]
        sp = []
        info = st.info.cpu().numpy() if form == "bsag" else None
        for w in range(P):
            if form == "bsag" and w == b:
                c = min(int(info[Q + b]), st.k_blk)
                sp += [one(c), st.sp_idx[w, b, :c], st.sp_val[w, b, :c]]
            else:
                sp += [st.sp_idx[w, b], st.sp_val[w, b]]
        out["sp"] = sp
        dr = []
        for i, m in enumerate(st.bags, start=1):
            cnt = st.drop_cnt[i - 1].cpu().numpy()
            for w in range(P):
                q = w % Q
                for t in range(m):
                    if (q + t) % Q == b:
                        c = int(cnt[w, t])
                        dr += [one(c), st.drop_idx[i - 1][w, t, :c], st.drop_val[i - 1][w, t, :c]]
        out["drops"] = dr
        if form == "rsag":
            sd = []
            for t in range(st.steps):
                sc = st.sag_cnt[t].cpu().numpy()
                for p in range(len(sc)):
                    j, q = divmod(p, Q)
                    if q != b:
                        continue
                    c = int(sc[p])
                    sd += [one(c), st.sag_idx[t][p, :c], st.sag_val[t][p, :c]]
            out["sag_drops"] = sd
        else:
            out["info"] = [torch.tensor([int(info[b]), int(info[Q + b])], dtype=torch.int32, device=st.dense.device)]
            tc = st.toph_cnt.cpu().numpy()
            th = []
            for tau in range(d):
                w = tau * Q + b
                c = int(tc[w])
                th += [one(c), st.toph_idx[w, :c], st.toph_val[w, :c]]
            out["toph_drops"] = th
    out["dense"] = [st.dense[lo:hi]]
    out["residual"] = [st.acc[w, lo:hi] for w in range(P)]
    return out


def host_digest(streams: dict) -> dict:
    out = {}
    for name, parts in streams.items():
        h = HostSum()
        for a in parts:
            h.add(a)
        out[name] = h.value()
    return out


def device_digest(streams: dict) -> dict:
    out = {}
    for name, parts in streams.items():
        h = DeviceSum()
        for a in parts:
            if a.numel():
                h.add(a)
        out[name] = h.value()
    return out
