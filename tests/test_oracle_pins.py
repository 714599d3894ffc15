"""Pins for the fp64 oracle: each test checks the oracle against something
other than itself -- hand-derived values, the paper's closed form solved by
LAPACK, its nilpotency lemma, sequential scans written in the paper's own
orientation, exhaustive tiny trees, and invariants that a dropped term, a
wrong sign, a wrong index or a transposed operand would break."""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from oracle import GDN, GLA

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# helpers written independently of the oracle (paper notation)
# --------------------------------------------------------------------------

def strict_ancestor_mask(parent):
    """M-_{ij} = 1[j in Anc(i)], built row by row from the parent's row
    (valid because every parent precedes its child)."""
    T = len(parent)
    M = np.zeros((T, T), dtype=bool)
    for i in range(T):
        p = parent[i]
        if p >= 0:
            M[i] = M[p]
            M[i, p] = True
    return M


def closed_form(mode, parent, Q, K, V, g, beta, S_pre):
    """Theorem 1 of §4.1 in the paper's orientation (S_pre is d_k x d_v):
    O = D_P Q S_pre + C (I+G)^{-1} D_beta (V - D_P K S_pre), with
    G = D_beta D_P [(K K^T) o M-] D_P^{-1} and C = D_P [(Q K^T) o M+] D_P^{-1}.
    For gated linear attention (u := v) the correction solve is dropped and
    U = V (Lemma 1's factorized readout)."""
    T = len(parent)
    Mm = strict_ancestor_mask(parent)
    Mp = Mm | np.eye(T, dtype=bool)
    gamma = np.exp(g)
    P = np.array([np.prod(gamma[Mp[i]]) for i in range(T)])
    DP, DPinv = np.diag(P), np.diag(1.0 / P)
    C = DP @ ((Q @ K.T) * Mp) @ DPinv
    B0 = DP @ Q @ S_pre
    if mode == GLA:
        U = V
    else:
        Db = np.diag(beta)
        G = Db @ DP @ ((K @ K.T) * Mm) @ DPinv
        R = Db @ (V - DP @ K @ S_pre)
        U = np.linalg.solve(np.eye(T) + G, R)       # LAPACK getrf/getrs
    return B0 + C @ U, U, P


def paper_scan(mode, Q, K, V, g, beta, S_pre):
    """Plain token-order recurrence of §2.1 Eq. gdn-background, S in
    R^{d_k x d_v}, o_t = S_t^T q_t."""
    S = S_pre.copy()
    out = []
    for t in range(Q.shape[0]):
        St = np.exp(g[t]) * S
        if mode == GLA:
            u = V[t]
        else:
            u = beta[t] * (V[t] - St.T @ K[t])
        S = St + np.outer(K[t], u)
        out.append(S.T @ Q[t])
    return np.array(out), S


def run_oracle(mode, parent, Q, K, V, g, beta, S_pre):
    """Single request, single head; S_pre in the paper's orientation."""
    T = len(parent)
    no = np.array([0, T], dtype=np.int32)
    st = S_pre.T[None, None]                     # stored orientation [1,1,dv,dk]
    O = oracle.verify(mode, 1, no, np.asarray(parent, np.int32), Q[:, None], K[:, None],
                      V[:, None], g[:, None], None if beta is None else beta[:, None], st)
    return O[:, 0]


def rand_case(rng, parent, dk, dv, mode):
    T = len(parent)
    Q = rng.standard_normal((T, dk))
    K = rng.standard_normal((T, dk))
    K /= np.linalg.norm(K, axis=1, keepdims=True)
    V = rng.standard_normal((T, dv))
    g = -np.logaddexp(0, rng.standard_normal(T))
    beta = 1 / (1 + np.exp(-rng.standard_normal(T))) if mode == GDN else None
    S_pre = 0.5 * rng.standard_normal((dk, dv))
    return Q, K, V, g, beta, S_pre


def random_parent(rng, T, roots=1):
    p = np.empty(T, dtype=np.int32)
    for i in range(T):
        p[i] = -1 if i < roots else rng.integers(0, i)
    return p


# --------------------------------------------------------------------------
# hand-derived values
# --------------------------------------------------------------------------

def test_appendix_scalar_values():
    spec = json.load(open(os.path.join(GOLDEN, "appendix_scalar.json")))
    trees = {}
    for c in spec["cases"]:
        mode = GLA if c["mode"] == "gla" else GDN
        parent = np.array(c["parent"], np.int32)
        T = len(parent)
        one = np.ones((T, 1))
        beta = None if c["beta"] is None else np.array(c["beta"], float)
        O = run_oracle(mode, parent, one, one, np.array(c["v"], float)[:, None],
                       np.full(T, np.log(0.5)), beta, np.ones((1, 1)))
        assert O[:, 0].tolist() == c["out"], c["name"]
        trees[c["name"]] = (mode, parent, c["v"], beta)
    for c in spec["commits"]:
        mode, parent, v, beta = trees[c["tree"]]
        T = len(parent)
        path = np.array(c["path"], np.int32)
        S = oracle.commit(mode, 1, np.array([0, T], np.int32), parent,
                          np.array([0, path.size], np.int32), path,
                          np.ones((T, 1, 1)), np.array(v, float)[:, None, None],
                          np.full((T, 1), np.log(0.5)),
                          None if beta is None else beta[:, None], np.ones((1, 1, 1, 1)))
        assert S[0, 0, 0, 0] == c["state"], c["name"]


# --------------------------------------------------------------------------
# the paper's own identities
# --------------------------------------------------------------------------

@pytest.mark.parametrize("mode", [GLA, GDN])
def test_chain_equals_token_order_scan(mode):
    rng = np.random.default_rng(1)
    dk, dv, T = 4, 8, 9                          # d_k != d_v: a transposition cannot pass
    parent = np.arange(-1, T - 1, dtype=np.int32)
    Q, K, V, g, beta, S_pre = rand_case(rng, parent, dk, dv, mode)
    ref, _ = paper_scan(mode, Q, K, V, g, beta, S_pre)
    np.testing.assert_allclose(run_oracle(mode, parent, Q, K, V, g, beta, S_pre), ref,
                               rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("mode", [GLA, GDN])
@pytest.mark.parametrize("seed", range(6))
def test_theorem1_closed_form(mode, seed):
    rng = np.random.default_rng(100 + seed)
    T = int(rng.integers(2, 48))
    parent = random_parent(rng, T, roots=1 + seed % 3)
    Q, K, V, g, beta, S_pre = rand_case(rng, parent, 6, 5, mode)
    ref, _, _ = closed_form(mode, parent, Q, K, V, g, beta, S_pre)
    np.testing.assert_allclose(run_oracle(mode, parent, Q, K, V, g, beta, S_pre), ref,
                               rtol=1e-10, atol=1e-11)


def test_nilpotency_and_neumann():
    """Lemma 3: G^{d+1} = 0 and (I+G)^{-1} = sum_{m<=d} (-G)^m; det(I+G) = 1."""
    rng = np.random.default_rng(7)
    for _ in range(10):
        T = int(rng.integers(3, 40))
        parent = random_parent(rng, T)
        Mm = strict_ancestor_mask(parent)
        d = int(Mm.sum(axis=1).max())
        # structural: boolean powers of the mask vanish at d+1, not before
        Pm = np.eye(T, dtype=np.int64)
        for m in range(1, d + 2):
            Pm = (Pm @ Mm.astype(np.int64)) > 0
            Pm = Pm.astype(np.int64)
            assert (Pm.sum() == 0) == (m == d + 1)
        Q, K, V, g, beta, S_pre = rand_case(rng, parent, 4, 3, GDN)
        gamma = np.exp(g)
        Mp = Mm | np.eye(T, dtype=bool)
        P = np.array([np.prod(gamma[Mp[i]]) for i in range(T)])
        G = np.diag(beta) @ np.diag(P) @ ((K @ K.T) * Mm) @ np.diag(1 / P)
        assert abs(np.linalg.det(np.eye(T) + G) - 1.0) < 1e-12
        R = rng.standard_normal((T, 3))
        U = R.copy()
        Z = R.copy()
        for _m in range(d):
            Z = -G @ Z
            U += Z
        np.testing.assert_allclose(U, np.linalg.solve(np.eye(T) + G, R), rtol=1e-11, atol=1e-12)
        ref, Uref, _ = closed_form(GDN, parent, Q, K, V, g, beta, S_pre)
        np.testing.assert_allclose(run_oracle(GDN, parent, Q, K, V, g, beta, S_pre), ref,
                                   rtol=1e-10, atol=1e-11)


@pytest.mark.parametrize("mode", [GLA, GDN])
def test_exhaustive_tiny_forests(mode):
    """Every parent array with T <= 5 (all labelled forests in
    parent-before-child order) against the closed form."""
    rng = np.random.default_rng(11)
    count = 0
    for T in range(1, 6):
        for parent in itertools.product(*[range(-1, i) for i in range(T)]):
            parent = np.array(parent, np.int32)
            Q, K, V, g, beta, S_pre = rand_case(rng, parent, 3, 2, mode)
            ref, _, _ = closed_form(mode, parent, Q, K, V, g, beta, S_pre)
            np.testing.assert_allclose(run_oracle(mode, parent, Q, K, V, g, beta, S_pre), ref,
                                       rtol=1e-10, atol=1e-12)
            count += 1
    assert count == 1 + 2 + 6 + 24 + 120


def test_gla_no_decay_no_prefix_is_masked_attention():
    """gamma = 1, S_pre = 0: gated linear attention reduces to the
    ancestor-masked (linear) attention ((Q K^T) o M+) V."""
    rng = np.random.default_rng(3)
    parent = random_parent(rng, 30, roots=2)
    Q, K, V, _, _, _ = rand_case(rng, parent, 5, 7, GLA)
    Mp = strict_ancestor_mask(parent) | np.eye(30, dtype=bool)
    ref = ((Q @ K.T) * Mp) @ V
    got = run_oracle(GLA, parent, Q, K, V, np.zeros(30), None, np.zeros((5, 7)))
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_zero_values_read_only_the_decayed_prefix():
    """V = 0 (GLA) or beta = 0 (GDN): o_i = P_i S_pre^T q_i."""
    rng = np.random.default_rng(4)
    parent = random_parent(rng, 25)
    for mode in (GLA, GDN):
        Q, K, V, g, beta, S_pre = rand_case(rng, parent, 6, 4, mode)
        if mode == GLA:
            V = np.zeros_like(V)
        else:
            beta = np.zeros_like(beta)
        Mp = strict_ancestor_mask(parent) | np.eye(25, dtype=bool)
        P = np.exp(np.array([g[Mp[i]].sum() for i in range(25)]))
        ref = P[:, None] * (Q @ S_pre)
        np.testing.assert_allclose(run_oracle(mode, parent, Q, K, V, g, beta, S_pre), ref,
                                   rtol=1e-12, atol=1e-13)


def test_delta_rule_with_unit_write_gate_recalls_value():
    """With beta = 1 and unit-norm k, the delta rule stores v exactly along
    k: S_i^T k_i = S~_i^T k_i + u_i (k_i^T k_i) = v_i.  So q_i = k_i gives
    o_i = v_i for every node, whatever S_pre and the gates are."""
    rng = np.random.default_rng(5)
    parent = random_parent(rng, 40, roots=3)
    Q, K, V, g, beta, S_pre = rand_case(rng, parent, 8, 6, GDN)
    got = run_oracle(GDN, parent, K, K, V, g, np.ones(40), S_pre)
    np.testing.assert_allclose(got, V, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------
# structural invariants
# --------------------------------------------------------------------------

@pytest.mark.parametrize("mode", [GLA, GDN])
def test_sibling_isolation(mode):
    """Perturbing node j's inputs changes exactly the outputs of j's subtree
    (the ancestor mask excludes siblings and descendants, §2.2)."""
    rng = np.random.default_rng(6)
    parent = random_parent(rng, 30)
    Q, K, V, g, beta, S_pre = rand_case(rng, parent, 5, 4, mode)
    base = run_oracle(mode, parent, Q, K, V, g, beta, S_pre)
    Mp = strict_ancestor_mask(parent) | np.eye(30, dtype=bool)
    for j in (0, 5, 17, 29):
        V2, g2 = V.copy(), g.copy()
        V2[j] += 1.0
        g2[j] -= 0.3
        out = run_oracle(mode, parent, Q, K, V2, g2, beta, S_pre)
        changed = np.abs(out - base).max(axis=1) > 1e-12
        np.testing.assert_array_equal(changed, Mp[:, j])


@pytest.mark.parametrize("mode", [GLA, GDN])
def test_relabelling_permutes_outputs(mode):
    rng = np.random.default_rng(8)
    T = 35
    parent = random_parent(rng, T, roots=2)
    Q, K, V, g, beta, S_pre = rand_case(rng, parent, 4, 5, mode)
    base = run_oracle(mode, parent, Q, K, V, g, beta, S_pre)
    # another topological order: repeatedly pick a random ready node
    ready = [i for i in range(T) if parent[i] < 0]
    order = []
    while ready:
        n = ready.pop(int(rng.integers(len(ready))))
        order.append(n)
        ready += [c for c in range(T) if parent[c] == n]
    new_of = {o: i for i, o in enumerate(order)}
    perm = np.array(order)
    parent2 = np.array([-1 if parent[o] < 0 else new_of[parent[o]] for o in order], np.int32)
    out = run_oracle(mode, parent2, Q[perm], K[perm], V[perm], g[perm],
                     None if beta is None else beta[perm], S_pre)
    np.testing.assert_allclose(out, base[perm], rtol=1e-12, atol=1e-13)


def test_gla_is_linear_in_values_and_prefix_state():
    rng = np.random.default_rng(9)
    parent = random_parent(rng, 20)
    Q, K, V1, g, _, S1 = rand_case(rng, parent, 4, 3, GLA)
    V2 = rng.standard_normal(V1.shape)
    S2 = rng.standard_normal(S1.shape)
    a = run_oracle(GLA, parent, Q, K, V1, g, None, S1)
    b = run_oracle(GLA, parent, Q, K, V2, g, None, S2)
    c = run_oracle(GLA, parent, Q, K, 2 * V1 - V2, g, None, 2 * S1 - S2)
    np.testing.assert_allclose(c, 2 * a - b, rtol=1e-11, atol=1e-12)


# --------------------------------------------------------------------------
# commit
# --------------------------------------------------------------------------

@pytest.mark.parametrize("mode", [GLA, GDN])
def test_commit_equals_accepted_commit_formula(mode):
    """Eq. accepted-commit (§4.4): S_new = P_a S_pre + (D_a K_a)^T U_a with
    U from the closed-form solve, and o_a = S_new^T q_a."""
    rng = np.random.default_rng(12)
    T = 40
    parent = random_parent(rng, T)
    Q, K, V, g, beta, S_pre = rand_case(rng, parent, 6, 4, mode)
    O, U, P = closed_form(mode, parent, Q, K, V, g, beta, S_pre)
    for a in (0, 7, 23, 39):
        path = []
        j = a
        while j >= 0:
            path.append(j)
            j = parent[j]
        path = path[::-1]
        Da = np.diag([P[a] / P[j] for j in path])
        S_new = P[a] * S_pre + (Da @ K[path]).T @ U[path]
        got = oracle.commit(mode, 1, np.array([0, T], np.int32), parent,
                            np.array([0, len(path)], np.int32), np.array(path, np.int32),
                            K[:, None], V[:, None], g[:, None],
                            None if beta is None else beta[:, None], S_pre.T[None, None])
        np.testing.assert_allclose(got[0, 0], S_new.T, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(got[0, 0] @ Q[a], O[a], rtol=1e-10, atol=1e-11)


def test_commit_empty_path_keeps_state_and_untouched_slots():
    rng = np.random.default_rng(13)
    parent = random_parent(rng, 10)
    Q, K, V, g, beta, S_pre = rand_case(rng, parent, 4, 4, GDN)
    state = rng.standard_normal((3, 1, 4, 4))
    got = oracle.commit(GDN, 1, np.array([0, 10], np.int32), parent,
                        np.array([0, 0], np.int32), np.zeros(0, np.int32),
                        K[:, None], V[:, None], g[:, None], beta[:, None], state,
                        slot=np.array([2], np.int32))
    np.testing.assert_array_equal(got, state)


@pytest.mark.parametrize("mode", [GLA, GDN])
def test_multistep_equals_grafted_tree(mode):
    """Committing path 1 and verifying tree 2 from the new state equals
    verifying tree 2 grafted below path 1's terminal node from the old one."""
    rng = np.random.default_rng(14)
    p1 = random_parent(rng, 12)
    Q1, K1, V1, g1, b1, S_pre = rand_case(rng, p1, 4, 5, mode)
    a = 11
    path = []
    j = a
    while j >= 0:
        path.append(j)
        j = p1[j]
    path = np.array(path[::-1], np.int32)
    S1 = oracle.commit(mode, 1, np.array([0, 12], np.int32), p1, np.array([0, path.size], np.int32),
                       path, K1[:, None], V1[:, None], g1[:, None],
                       None if b1 is None else b1[:, None], S_pre.T[None, None])
    p2 = random_parent(rng, 15, roots=2)
    Q2, K2, V2, g2, b2, _ = rand_case(rng, p2, 4, 5, mode)
    out2 = run_oracle(mode, p2, Q2, K2, V2, g2, b2, S1[0, 0].T)
    L = path.size
    chain = np.arange(-1, L - 1, dtype=np.int32)
    graft = np.concatenate([chain, np.where(p2 < 0, L - 1, p2 + L)]).astype(np.int32)
    cat = lambda x, y: None if x is None else np.concatenate([x[path], y])
    out = run_oracle(mode, graft, cat(Q1, Q2), cat(K1, K2), cat(V1, V2), cat(g1, g2),
                     cat(b1, b2), S_pre)
    np.testing.assert_allclose(out[L:], out2, rtol=1e-11, atol=1e-12)


# --------------------------------------------------------------------------
# topology and error classes
# --------------------------------------------------------------------------

def test_topology_masks_and_depths():
    rng = np.random.default_rng(15)
    sizes = [1, 5, 64, 65, 200, 256, 0, 3]
    parents = [random_parent(rng, T, roots=1 + (T > 50)) if T else np.zeros(0, np.int32)
               for T in sizes]
    parents[5] = np.arange(-1, 255, dtype=np.int32)           # a 256-node chain
    no = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    mask, depth = oracle.topology(no, np.concatenate(parents), 256)
    assert mask.shape == (sum(sizes), 4)
    for b, p in enumerate(parents):
        Mp = strict_ancestor_mask(p) | np.eye(len(p), dtype=bool)
        for i in range(len(p)):
            bits = [(int(mask[no[b] + i, j // 64]) >> (j % 64)) & 1 for j in range(256)]
            assert bits[:len(p)] == Mp[i].astype(int).tolist()
            assert not any(bits[len(p):])
            assert depth[no[b] + i] == Mp[i].sum() - 1


def test_error_classes():
    no = np.array([0, 3], np.int32)
    with pytest.raises(oracle.BadTree):
        oracle.check_forest(no, np.array([-1, 2, 0], np.int32), 8)      # parent after child
    with pytest.raises(oracle.BadTree):
        oracle.check_forest(no, np.array([-1, 1, 0], np.int32), 8)      # self parent
    with pytest.raises(oracle.BadTree):
        oracle.check_forest(no, np.array([-1, 0, 0], np.int32), 2)      # T_b > max_nodes
    with pytest.raises(oracle.BadTree):
        oracle.check_forest(np.array([0, 3, 2], np.int32), np.array([-1, 0, 0], np.int32), 8)
    p = np.array([-1, 0, 0], np.int32)
    ok = lambda path: oracle.check_paths(no, p, np.array([0, len(path)], np.int32),
                                         np.array(path, np.int32))
    ok([])
    ok([0, 2])
    for bad in ([1], [0, 1, 2], [0, 3], [2, 0], [0, -1]):
        with pytest.raises(oracle.BadPath):
            ok(bad)
    with pytest.raises(oracle.Unsupported):
        oracle.check_problem(1, 1, 1, 48, 128, 64, GLA)
    with pytest.raises(oracle.InvalidArg):
        oracle.check_problem(1, 3, 4, 128, 128, 64, GLA)
    with pytest.raises(oracle.Unsupported):
        oracle.check_problem(1, 1, 1, 128, 128, 257, GLA)


# --------------------------------------------------------------------------
# accepted path from a terminal node, and the cross-layer commit (§5.2)
# --------------------------------------------------------------------------

def test_accepted_paths_hand_derived():
    """P(a) = Anc(a) u {a}, root first, on trees whose paths are known by hand:
    a complete binary tree in BFS order (parent (i-1)//2), a chain, and a
    two-root forest; -1 is the empty path."""
    binary = np.array([-1] + [(i - 1) // 2 for i in range(1, 15)], np.int32)
    chain = np.arange(-1, 9, dtype=np.int32)
    forest = np.array([-1, 0, -1, 2, 3, 1, 3], np.int32)
    parent = np.concatenate([binary, chain, forest, binary])
    no = np.array([0, 15, 25, 32, 47], np.int32)
    offs, path = oracle.accepted_paths(no, parent, [14, 6, 6, -1])
    assert offs.tolist() == [0, 4, 11, 14, 14]
    assert path.tolist() == [0, 2, 6, 14] + [0, 1, 2, 3, 4, 5, 6] + [2, 3, 6]
    offs, path = oracle.accepted_paths(no, parent, [0, 9, 5, 7])
    assert path.tolist() == [0] + list(range(10)) + [0, 1, 5] + [0, 1, 3, 7]
    oracle.check_paths(no, parent, offs, path)


def test_accepted_paths_errors():
    no = np.array([0, 3], np.int32)
    p = np.array([-1, 0, 0], np.int32)
    for bad in (3, -2, 100):
        with pytest.raises(oracle.BadPath):
            oracle.accepted_paths(no, p, [bad])
    with pytest.raises(oracle.BadTree):
        oracle.accepted_paths(no, np.array([-1, 2, 0], np.int32), [1])
    with pytest.raises(oracle.InvalidArg):
        oracle.accepted_paths(no, p, [0, 1])


@pytest.mark.parametrize("mode", [GLA, GDN])
def test_commit_layers_is_each_layer_on_the_terminal_path(mode):
    """Three layers with their own rows and states, the path of each request
    written out by hand: every layer's result is the single-layer commit of
    that hand path, and a request with terminal -1 keeps its state."""
    rng = np.random.default_rng(16)
    binary = np.array([-1] + [(i - 1) // 2 for i in range(1, 15)], np.int32)
    parent = np.concatenate([binary, binary])
    no = np.array([0, 15, 30], np.int32)
    hand_offs = np.array([0, 4, 4], np.int32)
    hand_path = np.array([0, 1, 4, 9], np.int32)        # terminal 9 in request 0, none in 1
    layers = []
    for _ in range(3):
        k = rng.standard_normal((30, 2, 4))
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
        v = rng.standard_normal((30, 4, 4))
        g = -np.logaddexp(0.0, rng.standard_normal((30, 4)))
        beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((30, 4)))) if mode == GDN else None
        layers.append((k, v, g, beta, rng.standard_normal((2, 4, 4, 4))))
    got = oracle.commit_layers(mode, 2, no, parent, [9, -1], layers)
    for (k, v, g, beta, st), new in zip(layers, got):
        want = oracle.commit(mode, 2, no, parent, hand_offs, hand_path, k, v, g, beta, st)
        np.testing.assert_array_equal(new, want)
        np.testing.assert_array_equal(new[1], st[1])
        assert not np.allclose(new[0], st[0])


# --------------------------------------------------------------------------
# grouped heads and the query scale, against their definitions


def _grouped_case(rng, mode, Hk=2, Hv=6, dk=4, dv=3):
    parent = np.concatenate([random_parent(rng, 9), random_parent(rng, 7, roots=2)])
    node_offsets = np.array([0, 9, 16])
    N = parent.size
    q = rng.standard_normal((N, Hk, dk))
    k = rng.standard_normal((N, Hk, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((N, Hv, dv))
    g = -np.logaddexp(0, rng.standard_normal((N, Hv)))
    beta = 1 / (1 + np.exp(-rng.standard_normal((N, Hv)))) if mode == GDN else None
    state = 0.5 * rng.standard_normal((2, Hv, dv, dk))
    return node_offsets, parent, q, k, v, g, beta, state


@pytest.mark.parametrize("mode", [GLA, GDN])
def test_grouped_heads_equal_repeated_qk_heads(mode):
    """With Hk < Hv, each qk-head serves a run of Hv / Hk consecutive v-heads:
    the result equals the ungrouped computation (Hk = Hv) on q and k with
    every qk-head repeated that many times in place (numpy.repeat), for verify
    and for commit.  v, g, beta and the state stay per v-head.  Serving the
    groups the other way round (v-head h reading qk-head h mod Hk) differs."""
    rng = np.random.default_rng(21)
    Hk, Hv = 2, 6
    node_offsets, parent, q, k, v, g, beta, state = _grouped_case(rng, mode, Hk, Hv)
    rep = lambda t: np.repeat(t, Hv // Hk, axis=1)
    got = oracle.verify(mode, Hk, node_offsets, parent, q, k, v, g, beta, state)
    want = oracle.verify(mode, Hv, node_offsets, parent, rep(q), rep(k), v, g, beta, state)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)
    strided = lambda t: t[:, np.arange(Hv) % Hk]
    other = oracle.verify(mode, Hv, node_offsets, parent, strided(q), strided(k), v, g, beta, state)
    assert not np.allclose(got, other)
    path_offsets = np.array([0, 3, 5])
    path = np.array(oracle.root_path(parent[:9], 8)[:3] + oracle.root_path(parent[9:], 6)[:2])
    got = oracle.commit(mode, Hk, node_offsets, parent, path_offsets, path, k, v, g, beta, state)
    want = oracle.commit(mode, Hv, node_offsets, parent, path_offsets, path, rep(k), v, g, beta, state)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)
    assert not np.allclose(got, state)


@pytest.mark.parametrize("mode", [GLA, GDN])
def test_query_scale_scales_the_queries(mode):
    """q_scale multiplies the queries and nothing else: the readout is linear in
    q, so scaling by s equals reading out with s q at scale 1.  The state
    update (k, v, gates) does not see it."""
    rng = np.random.default_rng(22)
    node_offsets, parent, q, k, v, g, beta, state = _grouped_case(rng, mode)
    s = 0.37
    got = oracle.verify(mode, 2, node_offsets, parent, q, k, v, g, beta, state, q_scale=s)
    want = oracle.verify(mode, 2, node_offsets, parent, s * q, k, v, g, beta, state)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)
    assert not np.allclose(got, want / s)


def test_prefix_state_closed_forms():
    """The chain recurrence behind S_pre, against closed forms.  Gated linear
    attention: S_L = exp(sum g) S_0 + sum_t exp(sum_{s>t} g_s) v_t k_t^T.  Delta
    rule with g = 0, beta = 1 and orthonormal keys: every write replaces the
    value stored under its key, so S_L k_t = v_t for every t, and directions
    orthogonal to all keys read S_0."""
    rng = np.random.default_rng(23)
    L, U, dk, dv = 7, 2, 9, 5
    k = rng.standard_normal((L, U, dk))
    v = rng.standard_normal((L, U, dv))
    g = -np.logaddexp(0, rng.standard_normal((L, U)))
    S0 = rng.standard_normal((U, dv, dk))
    got = oracle.prefix_state(GLA, k, v, g, None, St0=S0)
    want = np.exp(g.sum(0))[:, None, None] * S0
    for t in range(L):
        w = np.exp(g[t + 1:].sum(0))[:, None, None]
        want = want + w * v[t][:, :, None] * k[t][:, None, :]
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.prefix_state(GLA, k, v, g, None),
                               want - np.exp(g.sum(0))[:, None, None] * S0, rtol=1e-12, atol=1e-12)

    basis = np.linalg.qr(rng.standard_normal((dk, dk)))[0]       # orthonormal columns
    keys = np.stack([basis[:, :L].T] * U, axis=1)                  # [L, U, dk]
    S = oracle.prefix_state(GDN, keys, v, np.zeros((L, U)), np.ones((L, U)), St0=S0)
    for t in range(L):
        np.testing.assert_allclose(np.einsum("uvk,uk->uv", S, keys[t]), v[t], atol=1e-12)
    x = basis[:, L]                                                 # orthogonal to every key
    np.testing.assert_allclose(S @ x, S0 @ x, atol=1e-12)
