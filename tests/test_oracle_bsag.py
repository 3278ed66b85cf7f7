"""Pins for the B-SAG step and the h controller of the CPU oracle (Sec. III-D,
Algorithm 2):

* Algorithm 2 traced by hand (tests/golden/bsag_controller_trace.json),
* the controller keeps h in [L/d, L] and drives N toward L on a monotone
  response,
* a pure-Python brute force of whole B-SAG steps (controller included) on
  tiny inputs, for several (P, d) with d not a power of 2 as well,
* conservation (update + residuals = inputs) exactly on dyadic inputs,
* identical teams: the union is d times one team's top-h,
* planted mistakes are caught.
"""

import json
import os

import numpy as np
import pytest

from oracle import spardl_oracle as so
from tests.bruteforce import bf_step_bsag
from tests.test_oracle import _rand_vals

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bits(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32)).view(np.uint32)


def _rows(rng, P, n, kind):
    if kind == "dyadic":
        return [rng.integers(-64, 65, size=n).astype(np.float32) for _ in range(P)]
    return [_rand_vals(rng, n, kind) for _ in range(P)]


def test_controller_hand_trace():
    g = json.load(open(os.path.join(GOLDEN, "bsag_controller_trace.json")))
    c = so.HController(g["L"], g["d"])
    for row in g["trace"]:
        c.observe(row["N_before"])
        cnt = c.next_count()
        assert (c.step, c.flag, c.h, cnt) == (row["step"], row["flag"], row["h"], row["count"]), row["why"]


def test_controller_range_and_direction():
    L, d = 1000, 7
    c = so.HController(L, d)
    for t in range(300):
        cnt = c.next_count()
        assert L / d <= c.h <= L and 1 <= cnt <= L
        c.observe(int(1.6 * cnt))          # union 1.6 x h: N = L needs h = 625
    assert abs(1.6 * c.h - L) < 0.05 * L
    c = so.HController(L, d)
    for t in range(50):
        c.next_count()
        c.observe(10 * L)                  # always too many: h sinks to its floor
    assert c.h == L / d


def _compare(P, d, n, L, steps, kind, seed):
    rng = np.random.default_rng(seed)
    acc_o = [np.zeros(n, np.float32) for _ in range(P)]
    acc_b = [np.zeros(n, np.float32) for _ in range(P)]
    c_o, c_b = {}, {}
    for t in range(steps):
        grad = _rows(rng, P, n, kind)
        u_bf, res_bf, final_bf, h_bf, N_bf = bf_step_bsag([a.copy() for a in acc_b], grad, P, L, d, c_b)
        acc_b = [np.array(r, np.float32) for r in res_bf]
        r = so.spardl_step_bsag(acc_o, grad, P, n, L, d, c_o)
        assert r.h == h_bf
        assert {q: len(r.union[q][0]) for q in r.blocks} == N_bf
        assert np.array_equal(bits(np.concatenate([r.dense[b] for b in r.blocks])), bits(u_bf))
        for w in range(P):
            assert np.array_equal(bits(acc_o[w]), bits(acc_b[w])), f"step {t} residual of worker {w}"
        for b in r.blocks:
            assert list(r.final[b][0]) == sorted(final_bf[b])


PD = [(2, 2), (3, 3), (6, 2), (6, 3), (8, 4), (9, 3), (10, 5), (12, 3), (14, 7)]


@pytest.mark.parametrize("P,d", PD)
@pytest.mark.parametrize("kind", ["normal", "ties", "dyadic"])
def test_matches_bruteforce(P, d, kind):
    Q = P // d
    rng = np.random.default_rng(900 + 13 * P + d + len(kind))
    n = int(rng.integers(4 * Q, 40 * Q + 1))
    min_len = min((b + 1) * n // Q - b * n // Q for b in range(Q))
    L = int(rng.integers(1, min_len + 1))
    _compare(P, d, n, L, 4, kind, 123 + P + d)


def test_controller_moves_in_whole_steps():
    """Large L: the controller's count changes over the steps, and the
    brute force follows it."""
    _compare(6, 3, 3000, 700, 8, "normal", 77)
    c, seen = {}, set()
    rng = np.random.default_rng(4)
    acc = [np.zeros(3000, np.float32) for _ in range(6)]
    for t in range(8):
        r = so.spardl_step_bsag(acc, _rows(rng, 6, 3000, "normal"), 6, 3000, 700, 3, c)
        seen.add(r.h[0])
    assert len(seen) > 3


@pytest.mark.parametrize("P,d", PD)
def test_conservation_dyadic(P, d):
    rng = np.random.default_rng(P * 29 + d)
    Q = P // d
    ctrl = {}
    n = int(rng.integers(Q, 30 * Q + 1))
    min_len = min((b + 1) * n // Q - b * n // Q for b in range(Q))
    L = int(rng.integers(1, min_len + 1))
    acc = [np.zeros(n, np.float32) for _ in range(P)]
    for t in range(4):
        grad = _rows(rng, P, n, "dyadic")
        A = [so.residual_add(a, g) for a, g in zip(acc, grad)]
        r = so.spardl_step_bsag(acc, grad, P, n, L, d, ctrl)
        u = np.concatenate([r.dense[b] for b in r.blocks]).astype(np.float64)
        lhs = u + np.sum(np.array(acc, dtype=np.float64), axis=0)
        assert np.array_equal(lhs, np.sum(np.array(A, dtype=np.float64), axis=0))
        for b in r.blocks:
            assert len(r.final[b][0]) == min(L, len(r.union[b][0]))
            assert len(r.union[b][0]) <= d * r.h[b]


@pytest.mark.parametrize("P,d", [(6, 3), (8, 2), (9, 9)])
def test_identical_teams(P, d):
    """Every team holds the same integer rows: each team's SRS ends the same,
    the union has the h indices of one team's top-h with d times its values."""
    rng = np.random.default_rng(P + d + 5)
    Q = P // d
    n = 20 * Q
    team = [rng.integers(-500, 501, size=n).astype(np.float32) for _ in range(Q)]
    grad = [team[w % Q].copy() for w in range(P)]
    acc = [np.zeros(n, np.float32) for _ in range(P)]
    r = so.spardl_step_bsag(acc, grad, P, n, 6, d, {})
    for q in r.blocks:
        ki, kv = r.kept_h[q]
        assert list(r.union[q][0]) == list(ki)
        assert np.array_equal(r.union[q][1], (kv.astype(np.float64) * d).astype(np.float32))


def test_planted_mistakes_are_caught(monkeypatch):
    def caught(fn):
        try:
            fn()
        except AssertionError:
            return True
        return False

    run = lambda: (_compare(6, 3, 90, 7, 3, "normal", 5), test_conservation_dyadic(6, 3), test_controller_hand_trace())
    run()
    # the controller without the xor: too many gradients drive h up
    orig = so.HController.next_count

    def no_xor(self):
        self.N = -self.N if self.N > self.L else self.N + 10 * self.L
        return orig(self)
    monkeypatch.setattr(so.HController, "next_count", no_xor)
    assert caught(run)
    monkeypatch.undo()
    # top-h drops not collected
    orig_sel = so.select_top
    calls = {"n": 0}

    def lose_drops(idx, val, c):
        ki, kv, di, dv = orig_sel(idx, val, c)
        return ki, kv, di[:0], dv[:0]
    monkeypatch.setattr(so, "select_top", lose_drops)
    assert caught(run)
    monkeypatch.undo()
    # N counted after the final top-L instead of after the gather
    orig_obs = so.HController.observe
    monkeypatch.setattr(so.HController, "observe", lambda self, N: orig_obs(self, min(N, self.L)))
    assert caught(lambda: _compare(6, 3, 3000, 700, 8, "normal", 77))
    monkeypatch.undo()
    run()
