"""Pins for the convolution front-end oracle (oracle/conv_oracle.py): each
test checks it against something other than itself -- numpy.convolve on a
chain, a hand-worked width-2 tree, hand-derived gate values, locality of the
window, and the commit composed with a later tree (grafting)."""
import numpy as np
import pytest

import oracle
import oracle.conv_oracle as co
from oracle import GDN, GLA


def silu(y):
    return y / (1.0 + np.exp(-y))


def case(rng, parent, Hk=1, Hv=2, dk=4, dv=4, width=4, slots=1):
    C = 2 * Hk * dk + Hv * dv
    N = len(parent)
    return dict(
        x=rng.standard_normal((N, C)), gate_a=rng.standard_normal((N, Hv)),
        gate_b=rng.standard_normal((N, Hv)), conv_weight=rng.standard_normal((C, width)),
        conv_bias=rng.standard_normal(C), A_log=rng.standard_normal(Hv) * 0.5,
        dt_bias=rng.standard_normal(Hv), conv_state=rng.standard_normal((slots, width - 1, C)))


def run(parent, d, mode=GDN, Hk=1, Hv=2, dk=4, dv=4, width=4, slot=None):
    T = len(parent)
    return oracle.conv_gates(mode, Hk, Hv, dk, dv, width, np.array([0, T]), np.asarray(parent),
                             d["x"], d["gate_a"], d["gate_b"] if mode == GDN else None,
                             d["conv_weight"], d["conv_bias"], d["A_log"], d["dt_bias"],
                             d["conv_state"], slot=slot)


@pytest.mark.parametrize("width", [2, 3, 4])
def test_chain_equals_numpy_convolve(width):
    """A chain is an ordinary token sequence: the causal depthwise convolution
    of (committed state rows, x rows) via numpy.convolve, then SiLU, then the
    per-head normalisation of q and k."""
    rng = np.random.default_rng(1)
    T, Hk, Hv, dk, dv = 9, 1, 2, 4, 4
    parent = np.arange(-1, T - 1)
    d = case(rng, parent, Hk, Hv, dk, dv, width)
    q, k, v, g, beta = run(parent, d, GDN, Hk, Hv, dk, dv, width)
    C = d["x"].shape[1]
    z = np.zeros((T, C))
    for c in range(C):
        seq = np.concatenate([d["conv_state"][0, :, c], d["x"][:, c]])
        y = np.convolve(seq, d["conv_weight"][c, ::-1], mode="valid")     # windows of `width`
        z[:, c] = silu(y + d["conv_bias"][c])
    qq = z[:, :Hk * dk].reshape(T, Hk, dk)
    kk = z[:, Hk * dk:2 * Hk * dk].reshape(T, Hk, dk)
    np.testing.assert_allclose(v, z[:, 2 * Hk * dk:].reshape(T, Hv, dv), rtol=1e-12, atol=1e-12)
    norm = lambda t: t / np.sqrt((t * t).sum(-1, keepdims=True) + 1e-6)   # the stated eps
    np.testing.assert_allclose(q, norm(qq), rtol=1e-12)
    np.testing.assert_allclose(k, norm(kk), rtol=1e-12)


def test_hand_worked_width_two_tree():
    """Width 2 with weights (1, 0) and zero bias: node i's pre-activation is
    its parent's input (the committed state row for a root)."""
    parent = np.array([-1, 0, 0, 1, -1])
    C = 2 * 1 * 2 + 1 * 2
    x = np.arange(5 * C, dtype=np.float64).reshape(5, C) / 10.0 - 1.0
    cs = np.full((1, 1, C), 0.25)
    Wt = np.tile([1.0, 0.0], (C, 1))
    q, k, v, g, beta = oracle.conv_gates(GLA, 1, 1, 2, 2, 2, np.array([0, 5]), parent, x,
                                         np.zeros((5, 1)), None, Wt, np.zeros(C), np.zeros(1),
                                         np.zeros(1), cs)
    want_pre = np.stack([cs[0, 0], x[0], x[0], x[1], cs[0, 0]])        # parent rows
    np.testing.assert_allclose(v.reshape(5, -1), silu(want_pre[:, 4:]), rtol=1e-13)
    assert beta is None


def test_gates_hand_values():
    """A_log = 0, dt_bias = 0, a = 0: g = -log 2; b = 0: beta = 1/2.  Large a:
    softplus(a) ~ a, so g ~ -exp(A_log) a."""
    parent = np.array([-1, 0])
    d = case(np.random.default_rng(2), parent)
    d["gate_a"][:] = 0.0
    d["gate_b"][:] = 0.0
    d["A_log"][:] = 0.0
    d["dt_bias"][:] = 0.0
    _, _, _, g, beta = run(parent, d)
    np.testing.assert_allclose(g, -np.log(2.0), rtol=1e-15)
    np.testing.assert_allclose(beta, 0.5, rtol=1e-15)
    d["gate_a"][:] = 40.0
    d["A_log"][:] = np.log(3.0)
    _, _, _, g, _ = run(parent, d)
    np.testing.assert_allclose(g, -3.0 * 40.0, rtol=1e-12)


def test_gates_bias_inside_softplus_and_signed_write_gate():
    """The bias shifts the softplus argument: head 0 has a = 1, dt_bias = -1, so
    softplus(0) = log 2; head 1 has a = 0, dt_bias = log(e - 1), so softplus = 1,
    and A_log = log 2 gives g = -2.  beta = sigmoid(b): b = log 3 gives 3/4,
    b = -log 3 gives 1/4."""
    parent = np.array([-1, 0, 0])
    d = case(np.random.default_rng(5), parent)
    d["gate_a"][:] = [1.0, 0.0]
    d["dt_bias"][:] = [-1.0, np.log(np.e - 1.0)]
    d["A_log"][:] = [0.0, np.log(2.0)]
    d["gate_b"][:] = [np.log(3.0), -np.log(3.0)]
    _, _, _, g, beta = run(parent, d)
    np.testing.assert_allclose(g[:, 0], -np.log(2.0), rtol=1e-14)
    np.testing.assert_allclose(g[:, 1], -2.0, rtol=1e-14)
    np.testing.assert_allclose(beta[:, 0], 0.75, rtol=1e-14)
    np.testing.assert_allclose(beta[:, 1], 0.25, rtol=1e-14)


def test_window_locality():
    """A node depends on its own input and its width-1 nearest ancestors only:
    changing a sibling, a descendant or an ancestor farther up leaves it
    unchanged, changing the parent does not."""
    rng = np.random.default_rng(3)
    parent = np.array([-1, 0, 1, 2, 3, 4, 3, 2])        # a chain 0..5 with side branches
    d = case(rng, parent, width=3)
    base = run(parent, d, width=3)
    node = 5                                           # window: nodes 3, 4, 5
    for other, changes in ((6, False), (7, False), (2, False), (1, False), (4, True), (3, True)):
        d2 = {kk: vv.copy() for kk, vv in d.items()}
        d2["x"][other] += 1.0
        out = run(parent, d2, width=3)
        same = all(np.allclose(a[node], b[node]) for a, b in zip(base[:3], out[:3]))
        assert same != changes, (other, changes)


def test_normalised_heads_and_slots():
    rng = np.random.default_rng(4)
    parent = np.array([-1, 0, 0, 1, 3])
    d = case(rng, parent, Hk=2, slots=3)
    q, k, *_ = run(parent, d, Hk=2, slot=np.array([2]))
    np.testing.assert_allclose(np.linalg.norm(q, axis=-1), 1.0, atol=1e-5)
    np.testing.assert_allclose(np.linalg.norm(k, axis=-1), 1.0, atol=1e-5)
    # the root's window uses slot 2's state, not slot 0's
    d2 = {kk: vv.copy() for kk, vv in d.items()}
    d2["conv_state"][0] += 5.0
    q2, *_ = run(parent, d2, Hk=2, slot=np.array([2]))
    np.testing.assert_array_equal(q, q2)


def test_state_commit_grafts():
    """Committing the path to node a and running a new tree from the new
    state equals running the new tree grafted below a from the old state."""
    rng = np.random.default_rng(5)
    width = 4
    p1 = np.array([-1, 0, 1, 0, 3, 4, 2])
    d = case(rng, p1, width=width)
    a = 5                                               # path 0, 3, 4, 5
    new = oracle.conv_state_commit(width, np.array([0, 7]), p1, [a], d["x"], d["conv_state"])
    np.testing.assert_array_equal(new[0], d["x"][[3, 4, 5]])
    short = oracle.conv_state_commit(width, np.array([0, 7]), p1, [3], d["x"], d["conv_state"])
    np.testing.assert_array_equal(short[0], np.concatenate([d["conv_state"][0, 2:], d["x"][[0, 3]]]))
    keep = oracle.conv_state_commit(width, np.array([0, 7]), p1, [-1], d["x"], d["conv_state"])
    np.testing.assert_array_equal(keep, d["conv_state"])
    p2 = np.array([-1, 0, -1, 2, 1])
    d2 = case(rng, p2, width=width)
    d2["conv_state"] = new
    out2 = run(p2, d2, width=width)
    path = [0, 3, 4, 5]
    graft_parent = np.concatenate([np.arange(-1, 3), np.where(p2 < 0, 3, p2 + 4)])
    dg = {kk: vv.copy() for kk, vv in d2.items()}
    for key in ("x", "gate_a", "gate_b"):
        dg[key] = np.concatenate([d[key][path], d2[key]])
    dg["conv_state"] = d["conv_state"]
    outg = run(graft_parent, dg, width=width)
    for a_, b_ in zip(out2, outg):
        np.testing.assert_allclose(a_, b_[4:], rtol=1e-12, atol=1e-12)


def test_errors():
    parent = np.array([-1, 0, 0])
    d = case(np.random.default_rng(6), parent)
    with pytest.raises(oracle.BadTree):
        run(np.array([-1, 2, 0]), d)
    with pytest.raises(oracle.InvalidArg):      # gate_b given to gated linear attention
        oracle.conv_gates(GLA, 1, 2, 4, 4, 4, np.array([0, 3]), parent, d["x"], d["gate_a"],
                          d["gate_b"], d["conv_weight"], d["conv_bias"], d["A_log"],
                          d["dt_bias"], d["conv_state"])
    for bad in (3, -2):
        with pytest.raises(oracle.BadPath):
            oracle.conv_state_commit(4, np.array([0, 3]), parent, [bad], d["x"], d["conv_state"])


def _window_off_by_one(conv_state_b, rows, width):
    seq = np.concatenate([conv_state_b, rows], axis=0)
    return np.concatenate([seq[-width - 1:-1]])[-width:] if seq.shape[0] > width else seq[-width:]


def _window_reversed(conv_state_b, rows, width):
    return np.concatenate([conv_state_b, rows], axis=0)[-width:][::-1]


@pytest.mark.parametrize("mut", [_window_off_by_one, _window_reversed])
def test_pins_reject_planted_window_mistakes(monkeypatch, mut):
    monkeypatch.setattr(co, "conv_window", mut)
    with pytest.raises(AssertionError):
        test_chain_equals_numpy_convolve(4)


# Gate mistakes are planted by editing the gate lines of a copy of the oracle's
# source; the copy is executed as a separate module, the oracle itself is untouched.
_GATE_LINE = "_softplus(a + np.asarray(dt_bias, np.float64)[None, :])"
_BETA_LINE = "_sigmoid(np.asarray(gate_b, np.float64))"
_GATE_MUTANTS = {
    "bias_outside_softplus": (_GATE_LINE, "(_softplus(a) + np.asarray(dt_bias, np.float64)[None, :])"),
    "bias_dropped": (_GATE_LINE, "_softplus(a)"),
    "write_gate_sign": (_BETA_LINE, "_sigmoid(-np.asarray(gate_b, np.float64))"),
}


@pytest.mark.parametrize("name", sorted(_GATE_MUTANTS))
def test_pins_reject_planted_gate_mistakes(monkeypatch, name):
    old, new = _GATE_MUTANTS[name]
    src = open(co.__file__).read()
    assert src.count(old) == 1
    mod = {"__name__": "oracle.conv_oracle_mutant", "__package__": "oracle"}
    exec(compile(src.replace(old, new), co.__file__, "exec"), mod)
    monkeypatch.setattr(oracle, "conv_gates", mod["conv_gates"])
    with pytest.raises(AssertionError):
        test_gates_bias_inside_softplus_and_signed_write_gate()
