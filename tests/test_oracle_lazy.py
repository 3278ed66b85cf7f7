"""Pins for the lazy-sparsification step of the CPU oracle (Sec. III-B
"Optimization for SRS", Algorithm 1):

* a step worked by hand (tests/golden/lazy_p2_worked.json), on which the lazy
  and eager steps give different updates,
* a pure-Python brute force of the lazy step on tiny inputs,
* closed forms: k/P = block length is an exact all-reduce with zero residual;
  identical integer workers give P * top-k; P = 1 is local top-k with local
  residual,
* conservation: final update + sum of residuals = sum of inputs, exactly on
  dyadic-integer inputs,
* running a subset of blocks is exact,
* planted mistakes in the oracle are caught by these pins.
"""

import json
import os

import numpy as np
import pytest

from oracle import spardl_oracle as so
from tests.bruteforce import bf_step_lazy
from tests.test_oracle import _rand_vals

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bits(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32)).view(np.uint32)


def _rows(rng, P, n, kind):
    if kind == "dyadic":
        return [rng.integers(-64, 65, size=n).astype(np.float32) for _ in range(P)]
    return [_rand_vals(rng, n, kind) for _ in range(P)]


def test_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "lazy_p2_worked.json")))
    P, n, k = g["P"], g["n"], g["k_per_block"]
    grad = [np.array(r, np.float32) for r in g["grad"]]
    acc = [np.array(r, np.float32) for r in g["residual_in"]]
    r = so.spardl_step_lazy(acc, grad, P, n, k)
    u = np.concatenate([r.dense[b] for b in range(P)])
    assert np.array_equal(bits(u), bits(g["lazy"]["update"]))
    for w in range(P):
        assert np.array_equal(bits(acc[w]), bits(g["lazy"]["residual"][w]))
    for key, idx in g["lazy"]["selections"].items():
        w, b = map(int, key.split(","))
        assert list(r.sel[(w, b)][0]) == idx
    acc_e = [np.array(r_, np.float32) for r_ in g["residual_in"]]
    e = so.spardl_step(acc_e, grad, P, n, k)
    assert np.array_equal(bits(np.concatenate([e.dense[b] for b in range(P)])), bits(g["eager"]["update"]))


def _compare_with_bruteforce(P, n, k, acc, grad):
    u_bf, res_bf, final_bf, sel_bf = bf_step_lazy([a.copy() for a in acc], grad, P, k)
    acc_o = [a.copy() for a in acc]
    r = so.spardl_step_lazy(acc_o, grad, P, n, k)
    u_o = np.concatenate([r.dense[b] for b in range(P)])
    assert np.array_equal(bits(u_o), bits(u_bf))
    for w in range(P):
        assert np.array_equal(bits(acc_o[w]), bits(res_bf[w])), f"residual of worker {w}"
    assert set(r.sel) == set(sel_bf)
    for key, (si, sv) in r.sel.items():
        assert list(si) == sorted(sel_bf[key])
        assert np.array_equal(bits(sv), bits([sel_bf[key][x] for x in sorted(sel_bf[key])]))
    for b in range(P):
        assert list(r.final[b][0]) == sorted(final_bf[b])


@pytest.mark.parametrize("P", [1, 2, 3, 4, 5, 6, 7, 8, 9])
@pytest.mark.parametrize("kind", ["normal", "ties", "dyadic"])
def test_matches_bruteforce(P, kind):
    rng = np.random.default_rng(3000 * P + len(kind))
    for trial in range(3):
        n = int(rng.integers(P, 64 + 1))
        min_len = min((b + 1) * n // P - b * n // P for b in range(P))
        k = int(rng.integers(1, min_len + 1))
        _compare_with_bruteforce(P, n, k, _rows(rng, P, n, kind), _rows(rng, P, n, kind))


@pytest.mark.parametrize("P", [2, 3, 4, 5, 6, 7, 8, 9, 12, 14])
def test_conservation_dyadic(P):
    """Final update + sum of new residuals = sum of inputs, at every index,
    exactly (partial sums of small integers are representable in fp32)."""
    rng = np.random.default_rng(P + 300)
    l = so.num_steps(P)
    for trial in range(5):
        n = int(rng.integers(P, 40 * P))
        min_len = min((b + 1) * n // P - b * n // P for b in range(P))
        k = int(rng.integers(1, min_len + 1))
        acc = _rows(rng, P, n, "dyadic")
        grad = _rows(rng, P, n, "dyadic")
        A = [so.residual_add(a, g) for a, g in zip(acc, grad)]
        r = so.spardl_step_lazy(acc, grad, P, n, k)
        u = np.concatenate([r.dense[b] for b in range(P)]).astype(np.float64)
        lhs = u + np.sum(np.array(acc, dtype=np.float64), axis=0)
        assert np.array_equal(lhs, np.sum(np.array(A, dtype=np.float64), axis=0))
        # every worker sparsifies every block exactly once, k entries each
        assert set(r.sel) == {(w, b) for w in range(P) for b in range(P)}
        assert all(len(si) == k for si, _ in r.sel.values())
        for (w, b), i in r.sent_at.items():
            assert i == (0 if b == w else next(s.i for s in so.srs_schedule(P) if b in s.sent_bag[w]))
            assert 0 <= i <= l


@pytest.mark.parametrize("P", [2, 3, 5, 8])
def test_full_density_is_exact_allreduce(P):
    rng = np.random.default_rng(P + 350)
    n, k = 12 * P, 12
    acc = _rows(rng, P, n, "dyadic")
    grad = _rows(rng, P, n, "dyadic")
    A = [so.residual_add(a, g) for a, g in zip(acc, grad)]
    r = so.spardl_step_lazy(acc, grad, P, n, k)
    u = np.concatenate([r.dense[b] for b in range(P)])
    assert np.array_equal(u.astype(np.float64), np.sum(np.array(A, np.float64), axis=0))
    for w in range(P):
        assert not np.any(acc[w])


@pytest.mark.parametrize("P", [2, 3, 4, 6, 7, 8])
def test_identical_integer_workers(P):
    """Every worker holds the same integer row: the final blocks are P times
    the local top-k (all partial sums exact), the residual is the row with the
    final indexes zeroed."""
    rng = np.random.default_rng(P + 377)
    n = 16 * P
    row = rng.integers(-1000, 1001, size=n).astype(np.float32)
    acc = [np.zeros(n, np.float32) for _ in range(P)]
    r = so.spardl_step_lazy(acc, [row.copy() for _ in range(P)], P, n, 5)
    bounds = so.block_bounds(n, P)
    for b in range(P):
        li, lv = so.local_sparsify(row[bounds[b]:bounds[b + 1]], bounds[b], 5)
        assert list(r.final[b][0]) == list(li)
        assert np.array_equal(r.final[b][1], (lv.astype(np.float64) * P).astype(np.float32))
    for w in range(P):
        expect = row.copy()
        for b in range(P):
            expect[r.final[b][0]] = 0.0
        assert np.array_equal(bits(acc[w]), bits(expect))


def test_single_worker_is_local_topk():
    rng = np.random.default_rng(8)
    n, k = 50, 7
    acc = [rng.standard_normal(n).astype(np.float32)]
    grad = [rng.standard_normal(n).astype(np.float32)]
    A = so.residual_add(acc[0], grad[0])
    r = so.spardl_step_lazy(acc, grad, 1, n, k)
    li, lv = so.local_sparsify(A, 0, k)
    dense = np.zeros(n, np.float32)
    dense[li] = lv
    assert np.array_equal(bits(r.dense[0]), bits(dense))
    expect = A.copy()
    expect[li] = 0.0
    assert np.array_equal(bits(acc[0]), bits(expect))


def test_block_subset_equals_full():
    rng = np.random.default_rng(6)
    P, n, k = 6, 600, 9
    acc = _rows(rng, P, n, "normal")
    grad = _rows(rng, P, n, "normal")
    acc_full = [a.copy() for a in acc]
    full = so.spardl_step_lazy(acc_full, grad, P, n, k)
    bounds = so.block_bounds(n, P)
    sub = [1, 4]
    acc_sub = [{b: acc[w][bounds[b]:bounds[b + 1]].copy() for b in sub} for w in range(P)]
    grad_sub = [{b: grad[w][bounds[b]:bounds[b + 1]] for b in sub} for w in range(P)]
    part = so.spardl_step_lazy(acc_sub, grad_sub, P, n, k, blocks=sub)
    for b in sub:
        assert np.array_equal(bits(part.dense[b]), bits(full.dense[b]))
        for w in range(P):
            assert np.array_equal(bits(acc_sub[w][b]), bits(acc_full[w][bounds[b]:bounds[b + 1]]))


def test_planted_mistakes_are_caught(monkeypatch):
    """Each plausible slip in the lazy oracle must fail at least one pin above."""
    rng = np.random.default_rng(98)
    P, n = 5, 60
    acc = _rows(rng, P, n, "dyadic")
    grad = _rows(rng, P, n, "dyadic")

    def caught(fn):
        try:
            fn()
        except AssertionError:
            return True
        return False

    def run():
        _compare_with_bruteforce(P, n, 3, [a.copy() for a in acc], grad)
        test_conservation_dyadic(P)
        test_worked_example()

    run()  # unmodified oracle passes

    orig = so.sparsify_with_residual
    orig_recv = so.add_received
    # xi that forgets to remove the selection
    monkeypatch.setattr(so, "sparsify_with_residual",
                        lambda G, base, k: orig(G, base, k)[:2] + (np.asarray(G, np.float32).copy(),))
    assert caught(run)
    monkeypatch.setattr(so, "sparsify_with_residual", orig)

    # summation that overwrites instead of adding: received values replace held ones
    def overwrite(G_block, base, idx, val):
        G_block[np.asarray(idx) - base] = val
    monkeypatch.setattr(so, "add_received", overwrite)
    assert caught(run)
    monkeypatch.setattr(so, "add_received", orig_recv)

    # a residual add that drops the carried residual
    orig_add = so.residual_add
    monkeypatch.setattr(so, "residual_add", lambda a, g: orig_add(g, np.zeros_like(g)))
    assert caught(lambda: _compare_with_bruteforce(P, n, 3, [a + 1 for a in acc], grad))
    monkeypatch.setattr(so, "residual_add", orig_add)

    # ties broken towards the higher index
    orig_topk = so.top_k
    monkeypatch.setattr(so, "top_k", lambda i, v, k: orig_topk(-np.asarray(i), v, k))
    assert caught(lambda: _compare_with_bruteforce(P, n, 3, _rows(np.random.default_rng(1), P, n, "ties"),
                                                   _rows(np.random.default_rng(2), P, n, "ties")))
    monkeypatch.setattr(so, "top_k", orig_topk)

    # sending to w - 2^(l-i) instead of w + 2^(l-i)
    orig_sched = so.srs_schedule

    def flipped(P_):
        return [so.SRSStep(st.i, st.distance, st.source, st.target, st.sent_bag,
                           tuple(tuple(st.sent_bag[t]) for t in st.target)) for st in orig_sched(P_)]
    monkeypatch.setattr(so, "srs_schedule", flipped)
    assert caught(run)
    monkeypatch.setattr(so, "srs_schedule", orig_sched)

    # the eager step in place of the lazy one
    monkeypatch.setattr(so, "spardl_step_lazy", lambda *a, **kw: _eager_as_lazy(*a, **kw))
    assert caught(test_worked_example)


def _eager_as_lazy(acc, grad, P, n, k, blocks=None):
    e = so.spardl_step(acc, grad, P, n, k, blocks)
    r = so.LazyStepResult(bounds=e.bounds, blocks=e.blocks)
    r.final, r.dense, r.residual = e.final, e.dense, e.residual
    r.sel = {(b, b): e.final[b] for b in e.blocks}
    return r
