"""Pins for the budget-allocation oracle (oracle/budget_oracle.py): a
hand-worked batch (with a tie and a per-request cap), brute-force optimality
of the selection on tiny forests, structural properties of the packed
forest, the error classes, and planted mistakes."""
import itertools

import numpy as np
import pytest

import oracle
import oracle.budget_oracle as bo
from synth import workloads as W


def hand_batch():
    # request 0: root r0; a (0.6), b (0.4) under r0; c (0.5), d (0.5) under a
    # request 1: root r1; e (0.9), f (0.1) under r1; g (0.5) under e
    parent = np.array([-1, 0, 0, 1, 1, -1, 0, 0, 1], np.int32)
    prob = np.array([1.0, 0.6, 0.4, 0.5, 0.5, 1.0, 0.9, 0.1, 0.5], np.float32)
    return np.array([0, 5, 9], np.int32), parent, prob


def test_hand_worked_selection():
    offs, parent, prob = hand_batch()
    # rho: a .6, b .4, c .3, d .3 | e .9, f .1, g .45 ; capacity 6 = 2 roots + e, a, g, b
    r = oracle.budget_select(offs, parent, prob, capacity=6, max_nodes=64)
    np.testing.assert_array_equal(r["rho"], np.float32([1, .6, .4, np.float32(.6) * np.float32(.5),
                                                        np.float32(.6) * np.float32(.5), 1, .9, .1,
                                                        np.float32(.9) * np.float32(.5)]))
    assert r["rank"].tolist() == [-1, 0, 1, 2, 3, -1, 0, 2, 1]
    assert r["node_offsets"].tolist() == [0, 3, 6]
    assert r["src"].tolist() == [0, 1, 2, 5, 6, 8]
    assert r["parent"].tolist() == [-1, 0, 0, -1, 0, 1]
    # one more node: c and d tie at .3; the lower candidate index (c) goes first
    r = oracle.budget_select(offs, parent, prob, capacity=7, max_nodes=64)
    assert r["src"].tolist() == [0, 1, 2, 3, 5, 6, 8]
    assert r["parent"].tolist() == [-1, 0, 0, 1, -1, 0, 1]


def test_per_request_cap():
    offs, parent, prob = hand_batch()
    r = oracle.budget_select(offs, parent, prob, capacity=6, max_nodes=2)
    assert r["node_offsets"].tolist() == [0, 2, 4]          # root + best child each; 2 slots unused
    assert r["src"].tolist() == [0, 1, 5, 6]


def test_capacity_covers_everything():
    offs, parent, prob = hand_batch()
    r = oracle.budget_select(offs, parent, prob, capacity=100, max_nodes=64)
    assert r["src"].tolist() == list(range(9))


def _feasible_best(offs, parent, rho, capacity, max_nodes):
    """Brute force: the largest achievable size and the best total rho over
    all selections that keep every root, are prefix-closed and respect the
    per-request cap."""
    B = len(offs) - 1
    M = int(offs[-1])
    nonroot = [v for v in range(M) if parent[v] != -1]
    roots = [v for v in range(M) if parent[v] == -1]
    req = np.repeat(np.arange(B), np.diff(offs))
    best = (-1, -1.0)
    for k in range(len(nonroot) + 1):
        for sub in itertools.combinations(nonroot, k):
            s = set(sub) | set(roots)
            if len(s) > capacity:
                continue
            if any(int(offs[req[v]]) + parent[v] not in s for v in sub):
                continue
            if any(sum(1 for v in s if req[v] == b) > max_nodes for b in range(B)):
                continue
            mass = sum(float(rho[v]) for v in s)
            best = max(best, (len(s), mass))
    return best


@pytest.mark.parametrize("seed", range(12))
def test_greedy_is_optimal_on_tiny_forests(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 4))
    parents, probs = [], []
    for _ in range(B):
        T = int(rng.integers(1, 6))
        par = np.array([-1] + [int(rng.integers(-1 if rng.random() < 0.15 else 0, i)) for i in range(1, T)],
                       np.int32)
        pr = rng.choice([0.125, 0.25, 0.5, 0.75, 1.0], T).astype(np.float32)   # ties happen
        parents.append(par)
        probs.append(pr)
    offs = np.concatenate([[0], np.cumsum([p.size for p in parents])]).astype(np.int32)
    parent, prob = np.concatenate(parents), np.concatenate(probs)
    nroots = int((parent == -1).sum())
    for capacity in range(nroots, int(offs[-1]) + 1):
        for max_nodes in (2, 3, 6):
            if any((p == -1).sum() > max_nodes for p in parents):
                continue
            r = oracle.budget_select(offs, parent, prob, capacity, max_nodes)
            size, mass = _feasible_best(offs, parent, r["rho"], capacity, max_nodes)
            got = r["src"]
            assert got.size == size
            assert abs(sum(float(r["rho"][v]) for v in got) - mass) < 1e-6


def test_packed_forest_properties():
    offs, parent, prob = W.make_candidates(3, [((8, 4, 2), 10), None, ((4, 4, 2), 8), ((16, 2), 6)],
                                           quantum=1 / 16)
    r = oracle.budget_select(offs, parent, prob, capacity=300, max_nodes=128)
    no, par, src, rho = r["node_offsets"], r["parent"], r["src"], r["rho"]
    assert no[-1] == 300 and no[2] == no[1]                 # full capacity; the empty request stays empty
    for b in range(len(no) - 1):
        T = no[b + 1] - no[b]
        assert T <= 128
        p = par[no[b]:no[b + 1]]
        s = src[no[b]:no[b + 1]]
        assert all(q == -1 or 0 <= q < i for i, q in enumerate(p))     # a forest, parent first
        assert np.all(np.diff(s) > 0)                                   # candidate order kept
        for i, q in enumerate(p):
            if q >= 0:
                assert parent[s[i]] == s[q] - offs[b]                   # same parent link
                assert rho[s[i]] <= rho[s[q]]
    # the selected set is a prefix of the batch-wide order (rho descending,
    # index ascending) restricted to eligible candidates: every eligible
    # candidate left out ranks after every selected non-root
    chosen = set(src.tolist())
    M = int(offs[-1])
    req = np.repeat(np.arange(len(offs) - 1), np.diff(offs))
    roots = np.array([int((parent[offs[b]:offs[b + 1]] == -1).sum()) for b in range(len(offs) - 1)])
    rank = r["rank"]
    assert all(v in chosen for v in range(M) if parent[v] == -1)        # every root kept
    assert all(rank[v] == -1 for v in range(M) if parent[v] == -1)
    eligible = [v for v in range(M) if parent[v] != -1 and rank[v] < 128 - roots[req[v]]]
    assert all(v in eligible for v in chosen if parent[v] != -1)        # only eligible ones taken
    key = lambda v: (-float(rho[v]), v)
    taken = [key(v) for v in eligible if v in chosen]
    left = [key(v) for v in eligible if v not in chosen]
    assert taken and left                                               # the case has both
    assert max(taken) < min(left)


def test_errors():
    offs, parent, prob = hand_batch()
    with pytest.raises(oracle.BadTree):
        bad = parent.copy()
        bad[3] = 4
        oracle.budget_select(offs, bad, prob, 6, 64)
    with pytest.raises(oracle.InvalidArg):
        oracle.budget_select(offs, parent, prob, 1, 64)            # two roots, capacity 1
    for bad_p in (1.5, -0.25, float("nan")):                       # not a probability
        bp = prob.copy()
        bp[2] = bad_p
        with pytest.raises(oracle.InvalidArg):
            oracle.budget_select(offs, parent, bp, 6, 64)


def test_pins_reject_a_flipped_tie_break(monkeypatch):
    monkeypatch.setattr(bo, "order_key", lambda rho, v: (-float(rho[v]), -v))
    with pytest.raises(AssertionError):
        test_hand_worked_selection()


def test_pins_reject_a_dropped_cap(monkeypatch):
    monkeypatch.setattr(bo, "room", lambda max_nodes, roots: 10 ** 6)
    with pytest.raises(AssertionError):
        test_per_request_cap()


def test_rho_rounds_at_every_step():
    """The stated reading: rho is the fp32 product formed root first, one
    rounding per step (on a long chain this differs from the exact product
    rounded once)."""
    par = np.arange(-1, 60, dtype=np.int32)
    p = np.float32(np.random.default_rng(0).uniform(0.5, 1.0, 61))
    step = [p[0]]
    for q in p[1:]:
        step.append(np.float32(step[-1] * q))
    exact_once = np.float32(np.cumprod(p.astype(np.float64)))
    assert not np.array_equal(np.float32(step), exact_once)     # the two readings differ here
    np.testing.assert_array_equal(bo.path_scores(par, p), np.float32(step))


def test_pins_reject_a_product_in_fp64(monkeypatch):
    def fp64_scores(cand_parent, cand_prob):
        r = np.zeros(len(cand_parent))
        for v, q in enumerate(cand_parent):
            r[v] = float(cand_prob[v]) if q == -1 else r[q] * float(cand_prob[v])
        return r.astype(np.float32)
    monkeypatch.setattr(bo, "path_scores", fp64_scores)
    with pytest.raises(AssertionError):
        test_rho_rounds_at_every_step()


# ----------------------------------------------------------------------------
# validity independent of rho's precision (tests/budget_validity.py): rho
# recomputed in fp64, the cut checked up to the fp32 rounding bound
# ----------------------------------------------------------------------------

from tests.budget_validity import check_selection  # noqa: E402


def _budget_batches():
    for name in ("tiny", "mid", "production", "gdn", "large"):
        case = W.budget_case(name)
        offs, par, prob = W.make_candidates(3, case.sizes)
        yield name, offs, par, prob, case.capacity, case.max_nodes
    sizes = [((3, 2), 5), None, ((4, 2, 1), 6), ((2,), 9), ((5, 3), 4), None, ((2, 2, 2), 7)]
    for quantum in (None, 1 / 16):
        offs, par, prob = W.make_candidates(11, sizes, quantum=quantum)
        roots = int((par == -1).sum())
        for max_nodes in (4, 16, 256):
            for capacity in (roots, roots + 7, roots + 40, int(offs[-1]) + 5):
                yield f"ties q={quantum} cap={max_nodes} C={capacity}", offs, par, prob, capacity, max_nodes


def test_oracle_selection_is_valid_at_any_precision():
    """The oracle's fp32 selection is a correct allocation under fp64 rho, up
    to the fp32 rounding bound (a pin that does not share the oracle's
    precision reading)."""
    for what, offs, par, prob, capacity, max_nodes in _budget_batches():
        r = oracle.budget_select(offs, par, prob, capacity, max_nodes)
        check_selection(offs, par, prob, capacity, max_nodes, r["node_offsets"], r["parent"], r["src"])


def test_validity_check_rejects_wrong_selections():
    """The check itself is not vacuous: swapping a selected node for a much
    weaker one, dropping a root, exceeding max_nodes, breaking candidate
    order or a parent link, or leaving capacity unused all fail it."""
    case = W.budget_case("production")
    offs, par, prob = W.make_candidates(3, case.sizes)
    r = oracle.budget_select(offs, par, prob, case.capacity, case.max_nodes)
    no, fpar, src = r["node_offsets"], r["parent"], r["src"]
    args = (offs, par, prob, case.capacity, case.max_nodes)
    check_selection(*args, no, fpar, src)
    rho = r["rho"]
    # a selected leaf of request 0 swapped for its request's weakest unselected leaf
    b0 = slice(no[0], no[1])
    s0 = src[b0]
    child_of = set(int(par[v]) + int(offs[0]) for v in s0 if par[v] >= 0)
    leaf = max((v for v in s0 if par[v] >= 0 and v not in child_of), key=lambda v: rho[v])
    cand = [v for v in range(offs[0], offs[1]) if v not in set(s0.tolist()) and par[v] >= 0
            and (par[v] + offs[0]) in set(s0.tolist()) and rho[v] < 0.5 * rho[leaf]]
    weak = min(cand, key=lambda v: rho[v])
    bad_src = src.copy()
    bad_par = fpar.copy()
    i_leaf = int(np.flatnonzero(s0 == leaf)[0])
    new = np.sort(np.concatenate([np.delete(s0, i_leaf), [weak]]))
    bad_src[b0] = new
    pos = {int(v): i for i, v in enumerate(new)}
    bad_par[b0] = [-1 if par[v] == -1 else pos[int(par[v] + offs[0])] for v in new]
    with pytest.raises(AssertionError):
        check_selection(*args, no, bad_par, bad_src)
    # a root dropped (request 1 keeps one node less, its first)
    with pytest.raises(AssertionError):
        check_selection(*args, no, fpar, np.concatenate([src[:no[1]], src[no[1] + 1:], src[-1:]]))
    # capacity left unused
    short = no.copy()
    short[-1] -= 1
    with pytest.raises(AssertionError):
        check_selection(*args, short, fpar, src)
    # candidate order broken inside a request
    swapped = src.copy()
    swapped[[no[2] + 1, no[2] + 2]] = swapped[[no[2] + 2, no[2] + 1]]
    with pytest.raises(AssertionError):
        check_selection(*args, no, fpar, swapped)
    # a parent link pointing at the wrong packed node
    relinked = fpar.copy()
    j = int(np.flatnonzero(fpar[no[3]:no[4]] > 0)[0]) + no[3]
    relinked[j] -= 1
    with pytest.raises(AssertionError):
        check_selection(*args, no, relinked, src)
    # a request over max_nodes
    with pytest.raises(AssertionError):
        check_selection(offs, par, prob, case.capacity, 8, no, fpar, src)
