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
    # a selected set is a prefix of the global order restricted to eligible nodes
    chosen = set(src.tolist())
    assert all(r["rank"][v] < 0 for v in range(int(offs[-1])) if parent[v] == -1 and v not in chosen) is True


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
