"""Plain CPU oracle of SparDL's sparse synchronisation with one team (d = 1).

TEST INFRASTRUCTURE ONLY -- see the package docstring.  Nothing in the product
path may import this module.

What is computed, and where the paper defines it (SparDL, arXiv 2304.00737):

* residual add: each worker adds its stored residual to its fresh gradient
  (Sec. III-B "Partitioning"; first step of Algorithm 1).
* partitioning into P blocks and l+1 bags (Sec. III-B "Partitioning",
  Example 1).
* block-wise top-k/P sparsification (Sec. III-B; top-k as defined in Sec. II
  "Top-k sparsification").
* Spar-Reduce-Scatter transmission: l = ceil(log2 P) steps; at step i worker w
  sends bag B_{l-i+1} to w + 2^{l-i} and receives the matching bag from
  w - 2^{l-i}, adds received entries into its held blocks by index and keeps
  the top k/P of every held block (Sec. III-B "Transmission with
  sparsification", Example 2, Theorem 1).
* final All-Gather of the P reduced blocks and decode to a dense update
  (end of Sec. III-B; Sec. II for All-Gather semantics).
* global residual collection (Sec. III-C, Algorithm 1).
* the lazy-sparsification variant of the transmission ("Optimization for
  SRS", Sec. III-B) with Algorithm 1's residual: held blocks stay dense,
  received entries are added into them, and a block is sparsified only when
  it is about to be sent (spardl_step_lazy; its own readings sit above it).

Readings taken where the paper is silent or ambiguous (each one is listed in
the design notes of the repository):

* fp32 throughout; every addition is one IEEE fp32 round-to-nearest-even add.
* top-k order: larger |v| first, compared on the fp32 bit pattern with the
  sign bit cleared; equal |v| -> lower index first.  Exactly k entries are kept
  (zeros and cancelled sums included) whenever at least k exist.
* blocks: block b covers [floor(b n / P), floor((b+1) n / P)).
* 0-based workers and blocks; worker w's preservation block is block w.
* eager sparsification: every block is sparsified locally before the first
  step and every held block that received entries is re-sparsified after each
  step (the variant the main text of Sec. III-B describes).
* residual collection: the in-procedure drops of one block at one worker over
  several steps are accumulated (not overwritten), in ascending step order,
  on top of the local residual.
* index sums add the held value and the received value (two operands; IEEE
  addition is commutative so operand order does not change the bits).

Arrays: values are numpy float32, indices numpy int64 (global indices within a
worker's flat gradient, i.e. in [0, n)).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# ----------------------------------------------------------------------------
# Partitioning and schedule (Sec. III-B "Partitioning", Example 1,
# "Transmission with sparsification", Example 2, Theorem 1)
# ----------------------------------------------------------------------------


def block_bounds(n: int, P: int) -> list[int]:
    """Start offsets of the P blocks plus the end: block b = [s_b, s_{b+1}).

    Sec. III-B splits the flat gradient into P blocks without saying how a
    remainder is spread; the reading used here is s_b = floor(b * n / P).
    """
    return [(b * n) // P for b in range(P + 1)]


def num_steps(P: int) -> int:
    """l = ceil(log2 P), the number of transmission steps (Sec. III-B); 0 for P = 1."""
    l = 0
    while (1 << l) < P:
        l += 1
    return l


def srs_partition_bags(P: int, w: int) -> list[list[int]]:
    """Bags B_0 .. B_l of worker w (Sec. III-B "Partitioning", Example 1).

    The P blocks are laid out on a circle starting at block w.  B_0 = {w} is
    the preservation bag; sending bag B_j takes the next 2^(j-1) blocks, and
    the last bag holds whatever remains (E = P - 2^(l-1) blocks).
    """
    l = num_steps(P)
    circle = [(w + t) % P for t in range(P)]
    bags = [circle[0:1]]
    pos = 1
    for j in range(1, l + 1):
        size = 1 << (j - 1)
        bags.append(circle[pos:pos + size])
        pos += size
    assert pos >= P and sum(len(b) for b in bags) == P
    return bags


@dataclass(frozen=True)
class SRSStep:
    """One transmission step i (1-based) of Spar-Reduce-Scatter."""

    i: int
    distance: int                 # 2^(l-i)
    target: tuple[int, ...]       # target[w] = w + distance (mod P)
    source: tuple[int, ...]       # source[w] = w - distance (mod P)
    sent_bag: tuple[tuple[int, ...], ...]      # blocks worker w sends at this step
    received_bag: tuple[tuple[int, ...], ...]  # blocks worker w receives at this step


def srs_schedule(P: int) -> list[SRSStep]:
    """The l transmission steps (Sec. III-B "Transmission with sparsification").

    At step i worker w sends its bag B_{l-i+1} to worker w + 2^(l-i) and
    receives bag B_{l-i+1} of worker w - 2^(l-i) (indices mod P).
    """
    l = num_steps(P)
    bags = [srs_partition_bags(P, w) for w in range(P)]
    steps = []
    for i in range(1, l + 1):
        dist = 1 << (l - i)
        j = l - i + 1
        target = tuple((w + dist) % P for w in range(P))
        source = tuple((w - dist) % P for w in range(P))
        sent = tuple(tuple(bags[w][j]) for w in range(P))
        recv = tuple(tuple(bags[source[w]][j]) for w in range(P))
        steps.append(SRSStep(i, dist, target, source, sent, recv))
    return steps


# ----------------------------------------------------------------------------
# Top-k sparsification (Sec. II "Top-k sparsification")
# ----------------------------------------------------------------------------


def magnitude_key(vals: np.ndarray) -> np.ndarray:
    """|v| as an unsigned integer: the fp32 bit pattern with the sign bit cleared.

    For finite floats this orders exactly like |v|, and it makes -0.0 and +0.0
    equal, as they are in magnitude.
    """
    v = np.ascontiguousarray(vals, dtype=np.float32)
    return v.view(np.uint32) & np.uint32(0x7FFFFFFF)


def top_k(idx: np.ndarray, vals: np.ndarray, k: int) -> np.ndarray:
    """Positions (into idx/vals) of the k entries with the largest |v|.

    Ties in |v| go to the lower index.  The positions are returned ordered by
    ascending index.  The selection uses one library primitive (a partial
    sort) on a combined key that is unique per entry: |v| in the high 32 bits
    and the complement of the index in the low 32 bits, so a larger combined
    key means "better" under exactly the order above.
    """
    m = len(idx)
    if k >= m:
        sel = np.arange(m)
    else:
        key = magnitude_key(vals).astype(np.uint64)
        comp = np.uint64(0xFFFFFFFF) - np.asarray(idx, dtype=np.uint64)
        combined = (key << np.uint64(32)) | comp
        sel = np.argpartition(combined, m - k)[m - k:]
    order = np.argsort(np.asarray(idx)[sel], kind="stable")
    return sel[order]


def local_sparsify(block_vals: np.ndarray, base: int, k: int) -> tuple[np.ndarray, np.ndarray]:
    """Top-k/P of one dense block (Sec. III-B): returns (global idx, val), idx ascending."""
    idx = np.arange(base, base + len(block_vals), dtype=np.int64)
    pos = top_k(idx, block_vals, k)
    return idx[pos], np.asarray(block_vals, dtype=np.float32)[pos].copy()


# ----------------------------------------------------------------------------
# Summation by index and re-sparsification (Sec. III-B; the SGA example of Sec. I)
# ----------------------------------------------------------------------------


def index_sum(h_idx, h_val, r_idx, r_val) -> tuple[np.ndarray, np.ndarray]:
    """Add received sparse entries into held sparse entries "according to the
    gradient indexes" (Sec. III-B): the union of both index sets, with
    held + received (one fp32 add) where an index is in both.  Sorted by index.
    """
    h_idx = np.asarray(h_idx, dtype=np.int64)
    r_idx = np.asarray(r_idx, dtype=np.int64)
    h_val = np.asarray(h_val, dtype=np.float32)
    r_val = np.asarray(r_val, dtype=np.float32)
    u_idx = np.union1d(h_idx, r_idx)
    u_val = np.empty(len(u_idx), dtype=np.float32)
    hp = np.searchsorted(u_idx, h_idx)
    rp = np.searchsorted(u_idx, r_idx)
    u_val[hp] = h_val
    in_both = np.isin(r_idx, h_idx)
    u_val[rp[~in_both]] = r_val[~in_both]
    u_val[rp[in_both]] = u_val[rp[in_both]] + r_val[in_both]
    return u_idx, u_val


def merge_and_resparsify(h_idx, h_val, r_idx, r_val, k: int):
    """Index-sum one received block into the held block, then keep its top k.

    Returns (kept_idx, kept_val, dropped_idx, dropped_val); both parts are
    sorted by index.  The dropped part is this worker's in-procedure residual
    for the block at this step (Sec. III-C).
    """
    u_idx, u_val = index_sum(h_idx, h_val, r_idx, r_val)
    keep = top_k(u_idx, u_val, k)
    mask = np.zeros(len(u_idx), dtype=bool)
    mask[keep] = True
    return u_idx[mask], u_val[mask], u_idx[~mask], u_val[~mask]


# ----------------------------------------------------------------------------
# The step (Algorithm 1 with d = 1)
# ----------------------------------------------------------------------------


def residual_add(acc: np.ndarray, grad: np.ndarray) -> np.ndarray:
    """G + xi in fp32 (first step of Algorithm 1)."""
    return (np.asarray(acc, dtype=np.float32) + np.asarray(grad, dtype=np.float32)).astype(np.float32)


def spar_reduce_scatter(S: dict, P: int, k: int, blocks=None):
    """Run the l transmission steps on the sparse blocks S[(w, b)] = (idx, val).

    Messages of step i carry the sender's blocks as they stood at the start of
    step i.  Only blocks in ``blocks`` (default: all) are processed; blocks never
    exchange data with one another, so restricting the set is exact.

    Returns drops[(i, w, b)] = (idx, val): what worker w discarded from block b
    at step i.  S is updated in place; S[(w, b)] keeps the state a block had
    when worker w sent it away.
    """
    wanted = set(range(P)) if blocks is None else set(blocks)
    held = [set(range(P)) for _ in range(P)]
    drops = {}
    for step in srs_schedule(P):
        sent_state = {}
        for w in range(P):
            for b in step.sent_bag[w]:
                assert b in held[w], "a sent block must still be held"
                if b in wanted:
                    sent_state[(w, b)] = S[(w, b)]
        for w in range(P):
            for b in step.sent_bag[w]:
                held[w].discard(b)
        for w in range(P):
            src = step.source[w]
            for b in step.received_bag[w]:
                # Theorem 1: every received block is still held by the receiver.
                assert b in held[w], "Theorem 1 violated"
                if b not in wanted:
                    continue
                h_idx, h_val = S[(w, b)]
                r_idx, r_val = sent_state[(src, b)]
                kept_i, kept_v, drop_i, drop_v = merge_and_resparsify(h_idx, h_val, r_idx, r_val, k)
                S[(w, b)] = (kept_i, kept_v)
                drops[(step.i, w, b)] = (drop_i, drop_v)
    for w in range(P):
        assert held[w] == {w}, "after l steps worker w holds only block w"
    return drops


def allgather_densify(final: dict, bounds: list[int], blocks) -> dict:
    """Dense update restricted to each listed block: the final value at every
    index that survived to the end of Spar-Reduce-Scatter, +0.0 elsewhere.
    The All-Gather gives every worker all P final blocks (Sec. III-B end), so
    the result is the same on every worker.
    """
    out = {}
    for b in blocks:
        dense = np.zeros(bounds[b + 1] - bounds[b], dtype=np.float32)
        idx, val = final[b]
        dense[np.asarray(idx) - bounds[b]] = val
        out[b] = dense
    return out


def global_residual_collect(A_block: np.ndarray, base: int, local_idx, final_idx, drops_in_order):
    """New residual of one worker on one block (Sec. III-C, Algorithm 1).

    Algorithm 1 keeps a copy of A = G + xi and, at every index I of the final
    global gradients, replaces the copy by what this worker discarded there.
    What worker w discarded at x is A[x] if w did not select x locally, 0 if it
    did, plus every in-procedure drop w made at x (in step order).  Indices
    outside I keep A[x]: local and end-procedure residuals stay where they
    arose.
    """
    xi = np.array(A_block, dtype=np.float32, copy=True)
    final_idx = np.asarray(final_idx, dtype=np.int64)
    L = np.asarray(local_idx, dtype=np.int64)
    L_in = L[np.isin(L, final_idx)]
    xi[L_in - base] = np.float32(0.0)
    for d_idx, d_val in drops_in_order:
        d_idx = np.asarray(d_idx, dtype=np.int64)
        m = np.isin(d_idx, final_idx)
        pos = d_idx[m] - base
        xi[pos] = xi[pos] + np.asarray(d_val, dtype=np.float32)[m]
    return xi


@dataclass
class SparDLStepResult:
    """Everything one oracle step produces, keyed by worker w and block b."""

    bounds: list
    blocks: list
    local: dict = field(default_factory=dict)    # (w, b) -> (idx, val) after local top-k
    S: dict = field(default_factory=dict)        # (w, b) -> (idx, val) after all steps
    drops: dict = field(default_factory=dict)    # (i, w, b) -> (idx, val)
    final: dict = field(default_factory=dict)    # b -> (idx, val) = S[(b, b)]
    dense: dict = field(default_factory=dict)    # b -> dense update on block b
    residual: dict = field(default_factory=dict)  # (w, b) -> new residual on block b


def _block_of(row, b, bounds):
    if isinstance(row, dict):
        return row[b]
    return row[bounds[b]:bounds[b + 1]]


def spardl_step(acc, grad, P: int, n: int, k: int, blocks=None) -> SparDLStepResult:
    """One SparDL synchronisation (d = 1) for P workers.

    acc[w], grad[w]: worker w's residual and fresh gradient, either full rows
    of length n or dicts {b: block array} holding at least the listed blocks.
    k is the per-block count k/P.  The new residual is written back into acc
    (in place) on the listed blocks; the result object holds the rest.
    """
    bounds = block_bounds(n, P)
    blocks = list(range(P)) if blocks is None else sorted(blocks)
    res = SparDLStepResult(bounds=bounds, blocks=blocks)
    A = {}
    for w in range(P):
        for b in blocks:
            A[(w, b)] = residual_add(_block_of(acc[w], b, bounds), _block_of(grad[w], b, bounds))
            res.local[(w, b)] = local_sparsify(A[(w, b)], bounds[b], k)
            res.S[(w, b)] = res.local[(w, b)]
    res.drops = spar_reduce_scatter(res.S, P, k, blocks)
    res.final = {b: res.S[(b, b)] for b in blocks}
    res.dense = allgather_densify(res.final, bounds, blocks)
    l = num_steps(P)
    for w in range(P):
        for b in blocks:
            in_order = [res.drops[(i, w, b)] for i in range(1, l + 1) if (i, w, b) in res.drops]
            xi = global_residual_collect(A[(w, b)], bounds[b], res.local[(w, b)][0],
                                         res.final[b][0], in_order)
            res.residual[(w, b)] = xi
            _block_of(acc[w], b, bounds)[...] = xi
    return res


# ----------------------------------------------------------------------------
# Lazy sparsification ("Optimization for SRS", Sec. III-B; Algorithm 1)
# ----------------------------------------------------------------------------
#
# Readings taken for this variant (each one is listed in the design notes):
#
# * a worker keeps every block it holds dense (A plus what it has received);
#   "the blocks transmitted next" at step i are the blocks of the bag sent at
#   step i, and they are sparsified right before that step's transmission;
#   the reserved block is sparsified after the last step.  So each worker
#   sparsifies each block exactly once.
# * summation adds each received entry into the receiver's dense block at its
#   index (one fp32 add, held + received); no re-selection follows it.
# * xi_b = G_b - g_b is an fp32 subtraction of a block that is zero off the
#   selection: G_b[x] off it (bits unchanged, -0.0 included), +0.0 on it.
# * I_b are the indexes of the final block b that the All-Gather delivers
#   (worker b's selection of its reserved block); the new residual of worker w
#   on block b is the copy of A taken before transmission, replaced on I_b by
#   worker w's xi_b.


@dataclass
class LazyStepResult:
    """Everything one lazy oracle step produces, keyed by worker w and block b."""

    bounds: list
    blocks: list
    sel: dict = field(default_factory=dict)       # (w, b) -> (idx, val): g_b as worker w selected it
    sent_at: dict = field(default_factory=dict)   # (w, b) -> step at which w sent b; 0 = reserved
    final: dict = field(default_factory=dict)     # b -> (idx, val) = sel[(b, b)]
    dense: dict = field(default_factory=dict)     # b -> dense update on block b
    residual: dict = field(default_factory=dict)  # (w, b) -> new residual on block b


def sparsify_with_residual(G_block: np.ndarray, base: int, k: int):
    """Top-k of one dense block and xi = G - g (Algorithm 1, sparsification
    and the residual line after it).  g is the selection written out densely
    (zeros elsewhere) and subtracted in fp32."""
    idx, val = local_sparsify(G_block, base, k)
    g = np.zeros(len(G_block), dtype=np.float32)
    g[idx - base] = val
    xi = (np.asarray(G_block, dtype=np.float32) - g).astype(np.float32)
    return idx, val, xi


def add_received(G_block: np.ndarray, base: int, idx, val) -> None:
    """Summation of a received sparse block into a dense held block (Sec. III-B,
    Algorithm 1 "transmission and summation"): one fp32 add per received index."""
    pos = np.asarray(idx, dtype=np.int64) - base
    G_block[pos] = G_block[pos] + np.asarray(val, dtype=np.float32)


def spardl_step_lazy(acc, grad, P: int, n: int, k: int, blocks=None) -> LazyStepResult:
    """One SparDL synchronisation (d = 1) with lazy sparsification: Algorithm 1
    as written, with the sparsification timing of "Optimization for SRS"
    (Sec. III-B).

    acc[w], grad[w]: as for spardl_step.  The new residual is written back into
    acc on the listed blocks.
    """
    bounds = block_bounds(n, P)
    blocks = list(range(P)) if blocks is None else sorted(blocks)
    wanted = set(blocks)
    res = LazyStepResult(bounds=bounds, blocks=blocks)
    # residual add, partition into blocks, and the copy of the result
    G, G_copy = {}, {}
    for w in range(P):
        for b in blocks:
            G[(w, b)] = residual_add(_block_of(acc[w], b, bounds), _block_of(grad[w], b, bounds))
            G_copy[(w, b)] = G[(w, b)].copy()
    xi = {}
    held = [set(range(P)) for _ in range(P)]
    for step in srs_schedule(P):
        # sparsify every block about to be sent, then send it
        for w in range(P):
            for b in step.sent_bag[w]:
                assert b in held[w], "a sent block must still be held"
                held[w].discard(b)
                if b in wanted:
                    idx, val, xi[(w, b)] = sparsify_with_residual(G[(w, b)], bounds[b], k)
                    res.sel[(w, b)] = (idx, val)
                    res.sent_at[(w, b)] = step.i
        # transmission and summation into the receivers' dense blocks
        for w in range(P):
            src = step.source[w]
            for b in step.received_bag[w]:
                assert b in held[w], "Theorem 1 violated"
                if b not in wanted:
                    continue
                add_received(G[(w, b)], bounds[b], *res.sel[(src, b)])
    for w in range(P):
        assert held[w] == {w}, "after l steps worker w holds only block w"
        if w in wanted:
            idx, val, xi[(w, w)] = sparsify_with_residual(G[(w, w)], bounds[w], k)
            res.sel[(w, w)] = (idx, val)
            res.sent_at[(w, w)] = 0
    res.final = {b: res.sel[(b, b)] for b in blocks}
    res.dense = allgather_densify(res.final, bounds, blocks)
    for w in range(P):
        for b in blocks:
            new = G_copy[(w, b)].copy()
            pos = res.final[b][0] - bounds[b]
            new[pos] = xi[(w, b)][pos]
            res.residual[(w, b)] = new
            _block_of(acc[w], b, bounds)[...] = new
    return res


# ----------------------------------------------------------------------------
# Spar-All-Gather across teams, recursive form (R-SAG; Sec. III-D, case "d is
# a power of 2")
# ----------------------------------------------------------------------------
#
# Readings taken for this part (each one is listed in the design notes):
#
# * team tau holds the consecutive workers tau Q .. tau Q + Q - 1, Q = P / d;
#   the worker at position q of its team runs SRS with its team (Q blocks of
#   the gradient, block b = [floor(b n / Q), floor((b+1) n / Q)), k_blk = L
#   entries per block) and ends holding block q.
# * at R-SAG step t (0-based, t < log2 d) team X exchanges with team X xor 2^t,
#   the partner at distance 2^t that is its own partner (recursive doubling);
#   the two workers at position q exchange block q, each adds the other's
#   entries by index (held + received, one fp32 add, the same on both sides)
#   and keeps the top L.
# * both sides drop the same entries.  At step t the two merged blocks are each
#   already held by 2^t workers (recursive doubling), so 2^(t+1) workers compute
#   the identical merge and drop the identical entries; each takes the share
#   2^-(t+1) of every dropped value into its residual (an exact fp32
#   multiplication by a power of two).  At the first step that is the half per
#   side that the paper states; after it, taking a half at every worker would
#   collect 2^t times what was dropped, so the share follows the paper's own
#   rule for B-SAG instead (1 / the number of workers holding the same copy).
#   Like the in-procedure drops of SRS these count at the final indices only,
#   after the SRS drops, in step order (elsewhere every worker keeps its own A).


def rsag_partner(X: int, t: int) -> int:
    """Team exchanging with team X at R-SAG step t (recursive doubling)."""
    return X ^ (1 << t)


@dataclass
class SagStepResult:
    """One step with d teams; blocks are the Q = P / d blocks of a worker."""

    bounds: list
    blocks: list
    local: dict = field(default_factory=dict)      # (w, b) -> (idx, val) after local top-L
    S: dict = field(default_factory=dict)          # (w, b) -> (idx, val) after SRS and SAG
    drops: dict = field(default_factory=dict)      # (i, w, b) -> (idx, val): SRS drops inside w's team
    sag_drops: dict = field(default_factory=dict)  # (t, w) -> (idx, val): what w's pair dropped of block w % Q
    final: dict = field(default_factory=dict)      # b -> (idx, val)
    dense: dict = field(default_factory=dict)
    residual: dict = field(default_factory=dict)


def sag_share(vals, t: int) -> np.ndarray:
    """A worker's share of the values its pair dropped at R-SAG step t: one
    fp32 multiplication by 2^-(t+1) (exact unless the result is subnormal)."""
    return (np.asarray(vals, dtype=np.float32) * np.float32(2.0 ** -(t + 1))).astype(np.float32)


def spardl_step_rsag(acc, grad, P: int, n: int, L: int, d: int, blocks=None) -> SagStepResult:
    """One SparDL synchronisation with d teams joined by R-SAG (Sec. III-D):
    SRS inside every team, log2 d recursive-doubling exchanges across teams
    with top-L after each, then the All-Gather inside the team; global
    residual collection over all three kinds of drops.

    L is the per-block count L(k, d, P) = d k / P.  acc / grad as for
    spardl_step, with the Q = P / d team blocks as the block structure.
    """
    assert d >= 1 and d & (d - 1) == 0 and P % d == 0, "R-SAG needs a power-of-two d dividing P"
    Q = P // d
    bounds = block_bounds(n, Q)
    blocks = list(range(Q)) if blocks is None else sorted(blocks)
    res = SagStepResult(bounds=bounds, blocks=blocks)
    A = {}
    for w in range(P):
        for b in blocks:
            A[(w, b)] = residual_add(_block_of(acc[w], b, bounds), _block_of(grad[w], b, bounds))
            res.local[(w, b)] = local_sparsify(A[(w, b)], bounds[b], L)
            res.S[(w, b)] = res.local[(w, b)]
    # SRS inside each team, on the team's own numbering
    for tau in range(d):
        Sq = {(q, b): res.S[(tau * Q + q, b)] for q in range(Q) for b in blocks}
        dr = spar_reduce_scatter(Sq, Q, L, blocks)
        for (q, b), v in Sq.items():
            res.S[(tau * Q + q, b)] = v
        for (i, q, b), v in dr.items():
            res.drops[(i, tau * Q + q, b)] = v
    # R-SAG across teams
    steps = d.bit_length() - 1
    for t in range(steps):
        for X in range(d):
            Y = rsag_partner(X, t)
            if Y < X:
                continue
            for q in blocks:
                wx, wy = X * Q + q, Y * Q + q
                hi, hv = res.S[(wx, q)]
                ri, rv = res.S[(wy, q)]
                ki, kv, di, dv = merge_and_resparsify(hi, hv, ri, rv, L)
                res.S[(wx, q)] = res.S[(wy, q)] = (ki, kv)
                res.sag_drops[(t, wx)] = res.sag_drops[(t, wy)] = (di, dv)
    for q in blocks:
        for X in range(1, d):
            assert np.array_equal(res.S[(X * Q + q, q)][0], res.S[(q, q)][0]), "teams disagree"
        res.final[q] = res.S[(q, q)]
    res.dense = allgather_densify(res.final, bounds, blocks)
    l = num_steps(Q)
    for w in range(P):
        for b in blocks:
            in_order = [res.drops[(i, w, b)] for i in range(1, l + 1) if (i, w, b) in res.drops]
            if b == w % Q:
                in_order += [(res.sag_drops[(t, w)][0], sag_share(res.sag_drops[(t, w)][1], t)) for t in range(steps)]
            xi = global_residual_collect(A[(w, b)], bounds[b], res.local[(w, b)][0], res.final[b][0], in_order)
            res.residual[(w, b)] = xi
            _block_of(acc[w], b, bounds)[...] = xi
    return res


# ----------------------------------------------------------------------------
# Spar-All-Gather across teams, Bruck form (B-SAG; Sec. III-D, case "d is not
# a power of 2") and the compression-ratio controller (Algorithm 2)
# ----------------------------------------------------------------------------
#
# Readings taken for this part (each one is listed in the design notes):
#
# * teams and the SRS inside them as for R-SAG; any d >= 2 dividing P.
# * every worker keeps the top h of the block it holds after SRS (h is the
#   controller's count for that block); what it drops is its own in-procedure
#   residual, collected in full.
# * the Bruck All-Gather hands every holder of block q the d top-h blocks; each
#   sums them by index in team order (((team 0 + team 1) + team 2) + ...), so
#   every team gets the same bits.  N_q is the number of distinct indices.
# * if N_q > L the holders keep the top L, otherwise all N_q stay.  The paper
#   gives each of the d holders 1/d of what this last selection drops; under
#   Algorithm 1's collection that share never reaches a residual (a dropped
#   index is not a final index, and off the final indices every worker keeps
#   its own A, which already accounts for the dropped values), so it is not
#   applied.  The same holds for the drops of R-SAG's last exchange.
# * Algorithm 2 runs per block q (all holders see the same N_q): state (h,
#   step, flag) in double precision, h = k/P = L/d, step = 0.01 (d - 1) L / d,
#   flag = false, and N = 0 before the first step.  At each step: if
#   (N > L) xor (step > 0) then (if flag: step = 2 step, flag = false; else
#   flag = true) else step = -step / 2, flag = false; h = h + step, clamped to
#   [L/d, L] (the range the paper gives for h); the count used is
#   floor(h + 1/2), clamped to [1, L].  N is then this step's N_q.


class HController:
    """Algorithm 2 for one block: the top-h count of each step."""

    def __init__(self, L: int, d: int):
        self.L, self.d = L, d
        self.lo = L / d
        self.h = self.lo
        self.step = 0.01 * (d - 1) * L / d
        self.flag = False
        self.N = 0

    def next_count(self) -> int:
        if (self.N > self.L) != (self.step > 0):
            if self.flag:
                self.step = self.step * 2.0
                self.flag = False
            else:
                self.flag = True
        else:
            self.step = -self.step * 0.5
            self.flag = False
        self.h = min(max(self.h + self.step, self.lo), float(self.L))
        return min(max(int(np.floor(self.h + 0.5)), 1), self.L)

    def observe(self, N: int) -> None:
        self.N = int(N)


@dataclass
class BsagStepResult:
    """One B-SAG step; blocks are the Q = P / d blocks of a worker."""

    bounds: list
    blocks: list
    h: dict = field(default_factory=dict)          # b -> top-h count used
    local: dict = field(default_factory=dict)      # (w, b) -> (idx, val) after local top-L
    S: dict = field(default_factory=dict)          # (w, b) -> (idx, val) after SRS
    drops: dict = field(default_factory=dict)      # (i, w, b) -> SRS drops inside w's team
    kept_h: dict = field(default_factory=dict)     # w -> (idx, val): top-h of the block w holds
    drop_h: dict = field(default_factory=dict)     # w -> (idx, val): the rest of it
    union: dict = field(default_factory=dict)      # b -> (idx, val): team-order sum of the top-h blocks
    final_drops: dict = field(default_factory=dict)  # b -> (idx, val) dropped by the final top-L
    final: dict = field(default_factory=dict)      # b -> (idx, val)
    dense: dict = field(default_factory=dict)
    residual: dict = field(default_factory=dict)


def select_top(idx, val, c: int):
    """Keep the top c of a sparse list (order of Sec. II / reading 4): returns
    (kept_idx, kept_val, dropped_idx, dropped_val), both by ascending index."""
    idx = np.asarray(idx, dtype=np.int64)
    val = np.asarray(val, dtype=np.float32)
    keep = top_k(idx, val, c)
    mask = np.zeros(len(idx), dtype=bool)
    mask[keep] = True
    return idx[mask], val[mask], idx[~mask], val[~mask]


def spardl_step_bsag(acc, grad, P: int, n: int, L: int, d: int, ctrl: dict, blocks=None) -> BsagStepResult:
    """One SparDL synchronisation with d teams joined by B-SAG (Sec. III-D):
    SRS inside every team, top-h, Bruck All-Gather across teams and summation,
    top-L, All-Gather inside the team; global residual collection over every
    kind of drop.  ctrl: {b: HController} carried across steps (created on
    first use)."""
    assert d >= 2 and P % d == 0
    Q = P // d
    bounds = block_bounds(n, Q)
    blocks = list(range(Q)) if blocks is None else sorted(blocks)
    res = BsagStepResult(bounds=bounds, blocks=blocks)
    A = {}
    for w in range(P):
        for b in blocks:
            A[(w, b)] = residual_add(_block_of(acc[w], b, bounds), _block_of(grad[w], b, bounds))
            res.local[(w, b)] = local_sparsify(A[(w, b)], bounds[b], L)
            res.S[(w, b)] = res.local[(w, b)]
    for tau in range(d):
        Sq = {(q, b): res.S[(tau * Q + q, b)] for q in range(Q) for b in blocks}
        dr = spar_reduce_scatter(Sq, Q, L, blocks)
        for (q, b), v in Sq.items():
            res.S[(tau * Q + q, b)] = v
        for (i, q, b), v in dr.items():
            res.drops[(i, tau * Q + q, b)] = v
    for q in blocks:
        c = ctrl.setdefault(q, HController(L, d)).next_count()
        res.h[q] = c
        for tau in range(d):
            w = tau * Q + q
            ki, kv, di, dv = select_top(*res.S[(w, q)], c)
            res.kept_h[w] = (ki, kv)
            res.drop_h[w] = (di, dv)
        ui, uv = res.kept_h[q]
        for tau in range(1, d):
            ui, uv = index_sum(ui, uv, *res.kept_h[tau * Q + q])
        res.union[q] = (ui, uv)
        ctrl[q].observe(len(ui))
        if len(ui) > L:
            ki, kv, di, dv = select_top(ui, uv, L)
        else:
            ki, kv, di, dv = ui, uv, ui[:0], uv[:0]
        res.final[q] = (ki, kv)
        res.final_drops[q] = (di, dv)
    res.dense = allgather_densify(res.final, bounds, blocks)
    l = num_steps(Q)
    for w in range(P):
        for b in blocks:
            in_order = [res.drops[(i, w, b)] for i in range(1, l + 1) if (i, w, b) in res.drops]
            if b == w % Q:
                in_order.append(res.drop_h[w])
            xi = global_residual_collect(A[(w, b)], bounds[b], res.local[(w, b)][0], res.final[b][0], in_order)
            res.residual[(w, b)] = xi
            _block_of(acc[w], b, bounds)[...] = xi
    return res
