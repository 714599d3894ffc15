"""The pins must be able to fail: plant plausible mistakes in the oracle's
update rule (on the CPU) and check that the pin tests reject every one."""
import numpy as np
import pytest

import oracle
import oracle.tree_oracle as to
from tests import test_oracle_pins as pins

_good_step = to.step


def _mut_decay_after_update(mode, St, k, v, g, beta):
    gamma = np.exp(g)[..., None, None]
    if mode == to.GLA:
        return gamma * (St + v[..., :, None] * k[..., None, :])
    return _good_step(mode, St, k, v, g, beta)


def _mut_delta_reads_undecayed(mode, St, k, v, g, beta):
    if mode == to.GLA:
        return _good_step(mode, St, k, v, g, beta)
    gamma = np.exp(g)[..., None, None]
    u = beta[..., None] * (v - np.einsum("...vk,...k->...v", St, k))
    return gamma * St + u[..., :, None] * k[..., None, :]


def _mut_delta_sign(mode, St, k, v, g, beta):
    if mode == to.GLA:
        return _good_step(mode, St, k, v, g, beta)
    gamma = np.exp(g)[..., None, None]
    u = beta[..., None] * (v + np.einsum("...vk,...k->...v", gamma * St, k))
    return gamma * St + u[..., :, None] * k[..., None, :]


def _mut_no_beta(mode, St, k, v, g, beta):
    if mode == to.GLA:
        return _good_step(mode, St, k, v, g, beta)
    return _good_step(mode, St, k, v, g, np.ones_like(beta))


def _mut_transposed_outer(mode, St, k, v, g, beta):
    gamma = np.exp(g)[..., None, None]
    return gamma * St + np.swapaxes(v[..., :, None] * k[..., None, :], -1, -2)


def _mut_gate_sign(mode, St, k, v, g, beta):
    return _good_step(mode, St, k, v, -g, beta)


MUTANTS = [_mut_decay_after_update, _mut_delta_reads_undecayed, _mut_delta_sign,
           _mut_no_beta, _mut_transposed_outer, _mut_gate_sign]

PIN_CHECKS = [
    pins.test_appendix_scalar_values,
    lambda: pins.test_chain_equals_token_order_scan(to.GLA),
    lambda: pins.test_chain_equals_token_order_scan(to.GDN),
    lambda: pins.test_theorem1_closed_form(to.GLA, 0),
    lambda: pins.test_theorem1_closed_form(to.GDN, 0),
    pins.test_delta_rule_with_unit_write_gate_recalls_value,
]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m.__name__)
def test_pins_reject_planted_mistake(mutant, monkeypatch):
    monkeypatch.setattr(to, "step", mutant)
    failures = 0
    for check in PIN_CHECKS:
        try:
            check()
        except (AssertionError, ValueError):
            failures += 1
    assert failures > 0, f"no pin caught {mutant.__name__}"


def test_pins_pass_unmutated():
    for check in PIN_CHECKS:
        check()
    assert oracle.step is _good_step


def _path_leaf_first(parent_b, i):
    out, j = [], int(i)
    while j != -1:
        out.append(j)
        j = int(parent_b[j])
    return out


def _path_without_terminal(parent_b, i):
    return _good_root_path(parent_b, i)[:-1]


def _path_without_root(parent_b, i):
    return _good_root_path(parent_b, i)[1:]


_good_root_path = to.root_path


@pytest.mark.parametrize("mut", [_path_leaf_first, _path_without_terminal, _path_without_root])
def test_path_pins_reject_planted_mistakes(monkeypatch, mut):
    monkeypatch.setattr(to, "root_path", mut)
    with pytest.raises((AssertionError, oracle.OracleError)):
        pins.test_accepted_paths_hand_derived()


# Mistakes outside the update step are planted by editing a copy of the
# oracle's source, executed as a separate module; the oracle is untouched.
_READOUT_LOOP = "            for t in root_path(pb, i):\n"
_VERIFY_HEADS = "    hq = np.arange(Hv) // grp                  # GQA"
_COMMIT_HEADS = "    hq = np.arange(Hv) // grp\n    new = state.copy()"
_SOURCE_MUTANTS = {
    "readout_before_own_update": [(_READOUT_LOOP, "            for t in root_path(pb, i)[:-1]:\n")],
    "heads_strided": [(_VERIFY_HEADS, "    hq = np.arange(Hv) % num_qk_heads  #"),
                      (_COMMIT_HEADS, "    hq = np.arange(Hv) % num_qk_heads\n    new = state.copy()")],
    "query_scale_dropped": [("O[o + i] = q_scale * np.einsum", "O[o + i] = np.einsum")],
    "query_scale_on_keys": [("O[o + i] = q_scale * np.einsum", "O[o + i] = np.einsum"),
                            ("St = step(mode, St, k[r, hq], v[r], g[r],\n                          None if beta is None else beta[r])\n            O",
                             "St = step(mode, St, q_scale * k[r, hq], v[r], g[r],\n                          None if beta is None else beta[r])\n            O")],
}

SOURCE_PIN_CHECKS = PIN_CHECKS + [
    lambda: pins.test_grouped_heads_equal_repeated_qk_heads(to.GLA),
    lambda: pins.test_grouped_heads_equal_repeated_qk_heads(to.GDN),
    lambda: pins.test_query_scale_scales_the_queries(to.GLA),
    lambda: pins.test_query_scale_scales_the_queries(to.GDN),
]


@pytest.mark.parametrize("name", sorted(_SOURCE_MUTANTS))
def test_pins_reject_planted_source_mistake(name, monkeypatch):
    src = open(to.__file__).read()
    for old, new in _SOURCE_MUTANTS[name]:
        assert src.count(old) == 1, old
        src = src.replace(old, new)
    mod = {"__name__": "oracle.tree_oracle_mutant", "__package__": "oracle"}
    exec(compile(src, to.__file__, "exec"), mod)
    for fn in ("verify", "commit"):
        monkeypatch.setattr(oracle, fn, mod[fn])
        monkeypatch.setattr(to, fn, mod[fn])
    failures = 0
    for check in SOURCE_PIN_CHECKS:
        try:
            check()
        except (AssertionError, ValueError):
            failures += 1
    assert failures > 0, f"no pin caught {name}"
