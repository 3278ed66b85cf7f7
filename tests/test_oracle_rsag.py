"""Pins for the R-SAG step of the CPU oracle (Sec. III-D, d a power of 2):

* a step worked by hand (tests/golden/rsag_p4_d4_worked.json) in which a drop
  shared by two teams lands on a final index, so the half shares matter,
* at d = 8 (three exchanges) a drop of the second exchange is shared by four
  workers; conservation pins the 2^-(t+1) share (a half at every step would
  collect it twice),
* a pure-Python brute force on tiny inputs, for several (P, d),
* d = 1 is the plain step; conservation (update + residuals = inputs) exactly
  on dyadic inputs; L = block length is an exact all-reduce with zero
  residual; every team ends with the same blocks,
* planted mistakes are caught.
"""

import json
import os

import numpy as np
import pytest

from oracle import spardl_oracle as so
from tests.bruteforce import bf_step_rsag
from tests.test_oracle import _rand_vals

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bits(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32)).view(np.uint32)


def _rows(rng, P, n, kind):
    if kind == "dyadic":
        return [rng.integers(-64, 65, size=n).astype(np.float32) for _ in range(P)]
    return [_rand_vals(rng, n, kind) for _ in range(P)]


def test_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "rsag_p4_d4_worked.json")))
    P, d, n, L = g["P"], g["d"], g["n"], g["L"]
    acc = [np.array(r, np.float32) for r in g["residual_in"]]
    grad = [np.array(r, np.float32) for r in g["grad"]]
    r = so.spardl_step_rsag(acc, grad, P, n, L, d)
    assert np.array_equal(bits(np.concatenate([r.dense[b] for b in r.blocks])), bits(g["update"]))
    for w in range(P):
        assert np.array_equal(bits(acc[w]), bits(g["residual"][w])), f"worker {w}"


def _compare(P, d, n, L, acc, grad):
    u_bf, res_bf, final_bf = bf_step_rsag([a.copy() for a in acc], grad, P, L, d)
    acc_o = [a.copy() for a in acc]
    r = so.spardl_step_rsag(acc_o, grad, P, n, L, d)
    assert np.array_equal(bits(np.concatenate([r.dense[b] for b in r.blocks])), bits(u_bf))
    for w in range(P):
        assert np.array_equal(bits(acc_o[w]), bits(res_bf[w])), f"residual of worker {w}"
    for b in r.blocks:
        assert list(r.final[b][0]) == sorted(final_bf[b])


PD = [(2, 2), (4, 2), (4, 4), (6, 2), (8, 2), (8, 4), (8, 8), (12, 4), (16, 8)]


@pytest.mark.parametrize("P,d", PD)
@pytest.mark.parametrize("kind", ["normal", "ties", "dyadic"])
def test_matches_bruteforce(P, d, kind):
    rng = np.random.default_rng(7000 + 31 * P + d + len(kind))
    Q = P // d
    for trial in range(2):
        n = int(rng.integers(Q, 48 + 1))
        min_len = min((b + 1) * n // Q - b * n // Q for b in range(Q))
        L = int(rng.integers(1, min_len + 1))
        _compare(P, d, n, L, _rows(rng, P, n, kind), _rows(rng, P, n, kind))


@pytest.mark.parametrize("P", [1, 2, 5, 8])
def test_one_team_is_the_plain_step(P):
    rng = np.random.default_rng(P + 400)
    n, L = 13 * P + 2, 3
    acc = _rows(rng, P, n, "normal")
    grad = _rows(rng, P, n, "normal")
    a1 = [a.copy() for a in acc]
    a2 = [a.copy() for a in acc]
    r1 = so.spardl_step_rsag(a1, grad, P, n, L, 1)
    r2 = so.spardl_step(a2, grad, P, n, L)
    for b in range(P):
        assert np.array_equal(bits(r1.dense[b]), bits(r2.dense[b]))
    for w in range(P):
        assert np.array_equal(bits(a1[w]), bits(a2[w]))


@pytest.mark.parametrize("P,d", PD)
def test_conservation_dyadic(P, d):
    rng = np.random.default_rng(P * 17 + d)
    Q = P // d
    for trial in range(4):
        n = int(rng.integers(Q, 30 * Q + 1))
        min_len = min((b + 1) * n // Q - b * n // Q for b in range(Q))
        L = int(rng.integers(1, min_len + 1))
        acc = _rows(rng, P, n, "dyadic")
        grad = _rows(rng, P, n, "dyadic")
        A = [so.residual_add(a, g) for a, g in zip(acc, grad)]
        r = so.spardl_step_rsag(acc, grad, P, n, L, d)
        u = np.concatenate([r.dense[b] for b in r.blocks]).astype(np.float64)
        lhs = u + np.sum(np.array(acc, dtype=np.float64), axis=0)
        assert np.array_equal(lhs, np.sum(np.array(A, dtype=np.float64), axis=0))
        for b in r.blocks:
            assert len(r.final[b][0]) == L
            for X in range(d):
                assert np.array_equal(r.S[(X * Q + b, b)][0], r.final[b][0])


@pytest.mark.parametrize("P,d", [(4, 2), (8, 4), (8, 8)])
def test_full_density_is_exact_allreduce(P, d):
    rng = np.random.default_rng(P + d + 90)
    Q = P // d
    n = 10 * Q
    acc = _rows(rng, P, n, "dyadic")
    grad = _rows(rng, P, n, "dyadic")
    A = [so.residual_add(a, g) for a, g in zip(acc, grad)]
    r = so.spardl_step_rsag(acc, grad, P, n, 10, d)
    u = np.concatenate([r.dense[b] for b in r.blocks])
    assert np.array_equal(u.astype(np.float64), np.sum(np.array(A, np.float64), axis=0))
    for w in range(P):
        assert not np.any(acc[w])
    assert all(len(di) == 0 for di, _ in r.sag_drops.values())


def test_planted_mistakes_are_caught(monkeypatch):
    rng = np.random.default_rng(55)
    P, d, n, L = 8, 4, 40, 3
    acc = _rows(rng, P, n, "dyadic")
    grad = _rows(rng, P, n, "dyadic")

    def caught(fn):
        try:
            fn()
        except AssertionError:
            return True
        return False

    def run():
        _compare(P, d, n, L, [a.copy() for a in acc], grad)
        test_worked_example()
        test_conservation_dyadic(P, d)

    run()
    # whole drops to both sides instead of half
    monkeypatch.setattr(so, "sag_share", lambda v, t: np.asarray(v, np.float32).copy())
    assert caught(run)
    monkeypatch.undo()
    # shared drops not collected at all
    monkeypatch.setattr(so, "sag_share", lambda v, t: np.zeros_like(np.asarray(v, np.float32)))
    assert caught(run)
    monkeypatch.undo()
    # a half at every step: with three exchanges the second one's drops are collected twice
    monkeypatch.setattr(so, "sag_share", lambda v, t: (np.asarray(v, np.float32) * np.float32(0.5)))
    assert caught(lambda: [test_conservation_dyadic(8, 8), test_conservation_dyadic(16, 8)])
    monkeypatch.undo()
    # partner at X + 2^t mod d instead of the recursive-doubling partner
    monkeypatch.setattr(so, "rsag_partner", lambda X, t: (X + (1 << t)) % 4)
    assert caught(run)
    monkeypatch.undo()
    run()
