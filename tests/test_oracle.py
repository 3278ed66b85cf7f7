"""Pins for the CPU oracle: checks against what the paper and mathematics fix.

* Example 1 / Example 2 / Theorem 1 of Sec. III-B (schedule),
* the reduce-scatter property (every worker ends with its own block, reduced
  over all P workers exactly once),
* the SGA growth example of Sec. I / Fig. 1 (3 + 3 entries -> 5),
* brute force (full sort, dict merges, a pure-Python step) on tiny inputs,
* closed forms: k/P = block length is an exact all-reduce with zero residual;
  identical workers give P * top-k; P = 1 is local top-k with local residual,
* conservation: final update + sum of residuals = sum of inputs, exactly on
  dyadic-integer inputs,
* planted mistakes in the oracle are caught by these pins.
"""

import json
import os
from collections import Counter

import numpy as np
import pytest

import oracle
from oracle import spardl_oracle as so
from tests.bruteforce import bf_merge, bf_step, bf_topk

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bits(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32)).view(np.uint32)


# --------------------------------------------------------------------------- schedule


def test_example1_partitioning():
    g = json.load(open(os.path.join(GOLDEN, "srs_examples_p6.json")))
    P, w = g["P"], g["worker"] - 1
    bags = so.srs_partition_bags(P, w)
    assert [[b + 1 for b in bag] for bag in bags] == g["bags"]
    assert so.num_steps(P) == g["l"]
    assert len(bags[-1]) == g["E"] == P - 2 ** (g["l"] - 1)


def test_example2_transmission():
    g = json.load(open(os.path.join(GOLDEN, "srs_examples_p6.json")))
    P, w = g["P"], g["worker"] - 1
    steps = so.srs_schedule(P)
    assert len(steps) == len(g["steps"])
    for st, ex in zip(steps, g["steps"]):
        assert st.i == ex["step"]
        assert st.distance == ex["distance"]
        assert st.target[w] + 1 == ex["sends_to"]
        assert len(st.sent_bag[w]) == ex["sent_blocks"]
        assert len(st.received_bag[w]) == ex["received_blocks"]
        src = st.source[w] + 1
        if ex["step"] == 1:
            # printed "2" contradicts the stated rule w - 2^(l-i); the rule gives 3
            assert ex["receives_from_printed"] == 2 and src == 3
        else:
            assert src == ex["receives_from_printed"]


@pytest.mark.parametrize("P", list(range(1, 130)))
def test_theorem1_and_reduce_scatter(P):
    """Theorem 1 (received bag within held blocks) and the reduce-scatter end
    state, by symbolic contributor multisets, for every P up to 129."""
    steps = so.srs_schedule(P)
    l = so.num_steps(P)
    assert len(steps) == l
    held = [set(range(P)) for _ in range(P)]
    contrib = {(w, b): Counter([w]) for w in range(P) for b in range(P)}
    sent_count = [0] * P
    for st in steps:
        snap = {key: Counter(c) for key, c in contrib.items()}
        for w in range(P):
            for b in st.sent_bag[w]:
                held[w].discard(b)
            sent_count[w] += len(st.sent_bag[w])
        for w in range(P):
            assert set(st.received_bag[w]) <= held[w]
            assert st.source[st.target[w]] == w
            assert list(st.received_bag[st.target[w]]) == list(st.sent_bag[w])
            for b in st.received_bag[w]:
                add = snap[(st.source[w], b)]
                assert not (set(contrib[(w, b)]) & set(add)), "a worker's data must not arrive twice"
                contrib[(w, b)] = contrib[(w, b)] + add
    for w in range(P):
        assert held[w] == {w}
        assert contrib[(w, w)] == Counter(range(P))
        assert sent_count[w] == P - 1  # Sec. III-B: every worker sends P-1 blocks


# --------------------------------------------------------------------------- top-k


def _rand_vals(rng, m, kind):
    if kind == "normal":
        return rng.standard_normal(m).astype(np.float32)
    if kind == "ties":
        v = rng.choice(np.array([0.0, 1.0, -1.0, 2.0, -2.0, 4.0, -4.0], dtype=np.float32), size=m)
        return (v * np.float32(2.0 ** -8)).astype(np.float32)
    if kind == "signed_zero":
        return rng.choice(np.array([0.0, -0.0, 1.0, -1.0], dtype=np.float32), size=m)
    raise ValueError(kind)


@pytest.mark.parametrize("kind", ["normal", "ties", "signed_zero"])
def test_topk_matches_full_sort(kind):
    rng = np.random.default_rng(7)
    for trial in range(200):
        m = int(rng.integers(1, 60))
        k = int(rng.integers(1, m + 1))
        vals = _rand_vals(rng, m, kind)
        base = int(rng.integers(0, 1000))
        idx, val = so.local_sparsify(vals, base, k)
        want = bf_topk({base + j: vals[j] for j in range(m)}, k)
        assert list(idx) == sorted(want.keys())
        assert np.array_equal(bits(val), bits([want[x] for x in sorted(want)]))


def test_topk_special_cases():
    v = np.full(37, -3.5, dtype=np.float32)
    idx, _ = so.local_sparsify(v, 100, 5)
    assert list(idx) == [100, 101, 102, 103, 104]          # equal |v|: lowest indices
    idx, val = so.local_sparsify(v, 0, 37)
    assert list(idx) == list(range(37))                      # k = length: identity
    z = np.array([0.0, -0.0, 0.0, -0.0], dtype=np.float32)
    idx, val = so.local_sparsify(z, 0, 2)
    assert list(idx) == [0, 1] and bits(val)[1] == 0x80000000  # -0 keeps its sign bit
    big = np.array([1.0, -8.0, 2.0, 8.0, -2.0], dtype=np.float32)
    idx, val = so.local_sparsify(big, 0, 3)
    assert list(idx) == [1, 2, 3] and list(val) == [-8.0, 2.0, 8.0]


# --------------------------------------------------------------------------- merge


def test_sga_example():
    """Sec. I / Fig. 1: worker 2 adds worker 1's 3 sparse gradients to its own 3
    and ends up with 5 (one shared index).  With k/P = 3 the block is cut back
    to 3 entries and the other 2 become in-procedure residual."""
    h_idx, h_val = np.array([2, 5, 9]), np.array([1.0, -3.0, 0.5], np.float32)
    r_idx, r_val = np.array([1, 5, 7]), np.array([2.0, 0.25, -4.0], np.float32)
    u_idx, u_val = so.index_sum(h_idx, h_val, r_idx, r_val)
    assert len(u_idx) == 5 and list(u_idx) == [1, 2, 5, 7, 9]
    assert u_val[2] == np.float32(-3.0) + np.float32(0.25)
    k_i, k_v, d_i, d_v = so.merge_and_resparsify(h_idx, h_val, r_idx, r_val, 3)
    assert list(k_i) == [1, 5, 7] and list(d_i) == [2, 9]
    assert len(k_i) == 3 and len(d_i) == 2


@pytest.mark.parametrize("kind", ["normal", "ties", "signed_zero"])
def test_merge_matches_dicts(kind):
    rng = np.random.default_rng(11)
    for trial in range(200):
        k = int(rng.integers(1, 12))
        universe = int(rng.integers(k, 3 * k + 2))
        hi = np.sort(rng.choice(universe, size=k, replace=False))
        ri = np.sort(rng.choice(universe, size=k, replace=False))
        hv, rv = _rand_vals(rng, k, kind), _rand_vals(rng, k, kind)
        k_i, k_v, d_i, d_v = so.merge_and_resparsify(hi, hv, ri, rv, k)
        merged = bf_merge(dict(zip(hi.tolist(), hv)), dict(zip(ri.tolist(), rv)))
        kept = bf_topk(merged, k)
        assert list(k_i) == sorted(kept) and len(k_i) == k
        assert np.array_equal(bits(k_v), bits([kept[x] for x in sorted(kept)]))
        dropped = sorted(set(merged) - set(kept))
        assert list(d_i) == dropped
        assert np.array_equal(bits(d_v), bits([merged[x] for x in dropped]))


# --------------------------------------------------------------------------- whole step


def _rows(rng, P, n, kind):
    if kind == "dyadic":
        return [rng.integers(-64, 65, size=n).astype(np.float32) for _ in range(P)]
    return [_rand_vals(rng, n, kind) for _ in range(P)]


def _compare_with_bruteforce(P, n, k, acc, grad):
    u_bf, res_bf, final_bf, drops_bf, local_bf = bf_step([a.copy() for a in acc], grad, P, k)
    acc_o = [a.copy() for a in acc]
    r = so.spardl_step(acc_o, grad, P, n, k)
    u_o = np.concatenate([r.dense[b] for b in range(P)])
    assert np.array_equal(bits(u_o), bits(u_bf))
    for w in range(P):
        assert np.array_equal(bits(acc_o[w]), bits(res_bf[w])), f"residual of worker {w}"
    for b in range(P):
        assert list(r.final[b][0]) == sorted(final_bf[b])
    assert set(r.drops) == {key for key, d in drops_bf.items()}
    for key, (di, dv) in r.drops.items():
        assert list(di) == sorted(drops_bf[key])
        assert np.array_equal(bits(dv), bits([drops_bf[key][x] for x in sorted(drops_bf[key])]))
    for (w, b), (li, lv) in r.local.items():
        assert list(li) == sorted(local_bf[(w, b)])


@pytest.mark.parametrize("P", [1, 2, 3, 4, 5, 6, 7, 8, 9])
@pytest.mark.parametrize("kind", ["normal", "ties", "dyadic"])
def test_step_matches_bruteforce(P, kind):
    rng = np.random.default_rng(1000 * P + len(kind))
    for trial in range(3):
        n = int(rng.integers(P, 64 + 1))
        min_len = min((b + 1) * n // P - b * n // P for b in range(P))
        k = int(rng.integers(1, min_len + 1))
        acc = _rows(rng, P, n, kind)
        grad = _rows(rng, P, n, kind)
        _compare_with_bruteforce(P, n, k, acc, grad)


@pytest.mark.parametrize("P", [2, 3, 4, 5, 6, 7, 8, 9, 12, 14])
def test_conservation_dyadic(P):
    """Final update + sum of new residuals = sum of inputs, at every index.
    Exact: every partial sum of small integers is representable in fp32."""
    rng = np.random.default_rng(P)
    for trial in range(5):
        n = int(rng.integers(P, 40 * P))
        min_len = min((b + 1) * n // P - b * n // P for b in range(P))
        k = int(rng.integers(1, min_len + 1))
        acc = _rows(rng, P, n, "dyadic")
        grad = _rows(rng, P, n, "dyadic")
        A = [so.residual_add(a, g) for a, g in zip(acc, grad)]
        r = so.spardl_step(acc, grad, P, n, k)
        u = np.concatenate([r.dense[b] for b in range(P)]).astype(np.float64)
        lhs = u + np.sum(np.array(acc, dtype=np.float64), axis=0)
        rhs = np.sum(np.array(A, dtype=np.float64), axis=0)
        assert np.array_equal(lhs, rhs)
        for b in range(P):                   # exactly k/P entries survive in every block
            assert len(r.final[b][0]) == k
        for (i, w, b), (di, dv) in r.drops.items():
            assert 0 <= len(di) <= k


@pytest.mark.parametrize("P", [2, 3, 5, 8])
def test_full_density_is_exact_allreduce(P):
    rng = np.random.default_rng(P + 50)
    n = 12 * P + 3
    k = min((b + 1) * n // P - b * n // P for b in range(P))
    if any((b + 1) * n // P - b * n // P != k for b in range(P)):
        n = 12 * P
        k = 12
    acc = _rows(rng, P, n, "dyadic")
    grad = _rows(rng, P, n, "dyadic")
    A = [so.residual_add(a, g) for a, g in zip(acc, grad)]
    r = so.spardl_step(acc, grad, P, n, k)
    u = np.concatenate([r.dense[b] for b in range(P)])
    assert np.array_equal(u.astype(np.float64), np.sum(np.array(A, np.float64), axis=0))
    for w in range(P):
        assert not np.any(acc[w])
    assert not r.drops or all(len(d[0]) == 0 for d in r.drops.values())


@pytest.mark.parametrize("P", [2, 3, 4, 6, 7, 8])
def test_identical_workers(P):
    rng = np.random.default_rng(P + 77)
    n = 16 * P
    row = rng.integers(-1000, 1001, size=n).astype(np.float32)
    acc = [np.zeros(n, np.float32) for _ in range(P)]
    grad = [row.copy() for _ in range(P)]
    r = so.spardl_step(acc, grad, P, n, 5)
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


def test_single_worker():
    rng = np.random.default_rng(3)
    n, k = 50, 7
    acc = [rng.standard_normal(n).astype(np.float32)]
    grad = [rng.standard_normal(n).astype(np.float32)]
    A = so.residual_add(acc[0], grad[0])
    r = so.spardl_step(acc, grad, 1, n, k)
    li, lv = so.local_sparsify(A, 0, k)
    assert list(r.final[0][0]) == list(li)
    dense = np.zeros(n, np.float32)
    dense[li] = lv
    assert np.array_equal(bits(r.dense[0]), bits(dense))
    expect = A.copy()
    expect[li] = 0.0
    assert np.array_equal(bits(acc[0]), bits(expect))
    assert r.drops == {}


def test_block_subset_equals_full():
    """Blocks never exchange data, so running only some of them is exact."""
    rng = np.random.default_rng(5)
    P, n, k = 6, 600, 9
    acc = _rows(rng, P, n, "normal")
    grad = _rows(rng, P, n, "normal")
    acc_full = [a.copy() for a in acc]
    full = so.spardl_step(acc_full, grad, P, n, k)
    bounds = so.block_bounds(n, P)
    sub = [1, 4]
    acc_sub = [{b: acc[w][bounds[b]:bounds[b + 1]].copy() for b in sub} for w in range(P)]
    grad_sub = [{b: grad[w][bounds[b]:bounds[b + 1]] for b in sub} for w in range(P)]
    part = so.spardl_step(acc_sub, grad_sub, P, n, k, blocks=sub)
    for b in sub:
        assert np.array_equal(bits(part.dense[b]), bits(full.dense[b]))
        for w in range(P):
            assert np.array_equal(bits(acc_sub[w][b]), bits(acc_full[w][bounds[b]:bounds[b + 1]]))


# --------------------------------------------------------------------------- planted mistakes


def test_planted_mistakes_are_caught(monkeypatch):
    """Each plausible slip in the oracle must fail at least one pin above."""
    rng = np.random.default_rng(99)
    P, n = 4, 40
    acc = _rows(rng, P, n, "ties")
    grad = _rows(rng, P, n, "ties")

    def caught(fn):
        try:
            fn()
        except AssertionError:
            return True
        return False

    run = lambda: _compare_with_bruteforce(P, n, 3, [a.copy() for a in acc], grad)
    run()  # unmodified oracle passes

    orig_topk = so.top_k
    # ties broken towards the higher index
    monkeypatch.setattr(so, "top_k", lambda i, v, k: orig_topk(-np.asarray(i), v, k))
    assert caught(run)
    monkeypatch.setattr(so, "top_k", orig_topk)

    # merge that keeps the received value instead of adding it
    orig_sum = so.index_sum

    def bad_sum(hi, hv, ri, rv):
        u_i, u_v = orig_sum(hi, hv, ri, np.zeros_like(rv))
        u_i2, u_v2 = orig_sum(ri, rv, hi, np.zeros_like(hv))
        return u_i, np.where(np.isin(u_i, ri), u_v2, u_v).astype(np.float32)
    monkeypatch.setattr(so, "index_sum", bad_sum)
    assert caught(run)
    monkeypatch.setattr(so, "index_sum", orig_sum)

    # residual collection that forgets the in-procedure drops
    orig_grc = so.global_residual_collect
    monkeypatch.setattr(so, "global_residual_collect",
                        lambda A, base, L, F, d: orig_grc(A, base, L, F, []))
    assert caught(run)
    monkeypatch.setattr(so, "global_residual_collect", orig_grc)

    # sending to w - 2^(l-i) instead of w + 2^(l-i)
    orig_sched = so.srs_schedule

    def flipped(P_):
        out = []
        for st in orig_sched(P_):
            out.append(so.SRSStep(st.i, st.distance, st.source, st.target,
                                  st.sent_bag, tuple(tuple(st.sent_bag[t]) for t in st.target)))
        return out
    monkeypatch.setattr(so, "srs_schedule", flipped)
    assert caught(run)
    monkeypatch.setattr(so, "srs_schedule", orig_sched)
