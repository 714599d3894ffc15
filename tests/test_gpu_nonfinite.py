"""Where a non-finite input (NaN or Inf) can reach, through the C ABI.

A NaN or Inf in one request's q, k, v, g, beta or state slot is compared with
a clean run of the same batch:
* it never reaches another request's outputs or state slot, nor a v-head
  outside the affected group (bit-identical to the clean run);
* it reaches at least what the sequential definition says (§4.1): the node
  itself for q; the node's subtree for k, v, g and beta; every node of the
  request for the state;
* it reaches at most: the node for q; the subtree for k and g under gated
  linear attention (ancestor masking is a select, so the masked
  coefficients stay exactly zero); every node of the request for the state,
  for v under gated linear attention and for k, v, g and beta under the
  delta rule.  These go wider than the definition because the on-chip
  contractions run over whole 16-node tiles: a non-finite v (or, under the
  delta rule, u) times the zero coefficient of a non-descendant is NaN in
  IEEE arithmetic;
* the commit reads only the accepted path's rows: a non-finite node off the
  path leaves the slot bit-identical to the clean commit, one on it (or a
  non-finite state entry) makes the affected heads' slots non-finite, and
  other slots are never touched.
"""
import dataclasses

import numpy as np
import pytest

from synth import workloads as W
from tests import gpu_helpers as H
from tests.test_gpu_edge import cfg_of, chain_path, custom, rand_state

pytestmark = pytest.mark.gpu

CASES = {   # name: (base config, rule, node cap, tree sizes of the 3 requests)
    "small": ("production", W.GLA, 64, [30, 40, 25]),
    "tiled": ("large", W.GLA, 256, [100, 150, 70]),
    "gdn": ("gdn", W.GDN, 128, [90, 128, 60]),
    "gdn_wide": ("gdn", W.GDN, 256, [100, 200, 30]),
}
HK, HV = 2, 4


def _subtree(parent, j):
    """j and its descendants: the nodes whose root path holds j."""
    return [i for i in range(len(parent)) if j in W.path_to(parent, i)]


def _setup(case):
    base, mode, cap, sizes = CASES[case]
    cfg = cfg_of(base, batch=3, mode=mode, prefix_len=0, max_nodes=cap, num_qk_heads=HK, num_v_heads=HV)
    rng = np.random.default_rng([cap, mode])
    parents = [W.topk_tree(rng, T, (4, 3, 2), 12) for T in sizes]
    p1 = parents[1]
    # node j of request 1: a child of the root with a subtree of several nodes
    kids = [i for i in range(len(p1)) if p1[i] == 0]
    j = max(kids, key=lambda c: len(_subtree(p1, c)))
    sub = _subtree(p1, j)
    other = next(c for c in kids if c != j)
    deep_on = max(sub, key=lambda i: len(W.path_to(p1, i)))
    off = [i for i in range(len(p1)) if i not in sub]
    deep_off = max(off, key=lambda i: len(W.path_to(p1, i)))
    assert other in off
    return cfg, parents, j, sub, deep_on, deep_off


def _run(cfg, w, state):
    up = H.Uploaded(w)
    out, err = H.run_verify(cfg, up, H.t_f32(state))
    assert err == 0
    st = H.t_f32(state)
    assert H.run_commit(cfg, up, st) == 0
    return out, st.cpu().numpy()


KINDS = ["q", "k", "v", "g", "beta", "state"]
PARAMS = [(c, k, on) for c in CASES for k in KINDS for on in (True, False)
          if k != "beta" or CASES[c][1] == W.GDN]   # beta exists under the delta rule only


@pytest.mark.parametrize("case, kind, on_path", PARAMS)
def test_nonfinite_reach(case, kind, on_path):
    cfg, parents, j, sub, deep_on, deep_off = _setup(case)
    gdn = cfg.mode == W.GDN
    paths = [chain_path(p, len(p) - 1) for p in parents]
    paths[1] = chain_path(parents[1], deep_on if on_path else deep_off)
    w = custom(cfg, parents, paths, seed=5)
    state = rand_state(cfg, 3, seed=5)
    out_c, st_c = _run(cfg, w, state)
    assert np.isfinite(out_c).all() and np.isfinite(st_c).all()

    o1 = int(w.node_offsets[1])
    rj = o1 + j
    hq, h = 1, 2                        # the poisoned qk-head, and v-head (in qk-head 1's group)
    group = [x for x in range(HV) if x // (HV // HK) == hq]
    bad = np.nan if kind in ("q", "k", "g", "beta") else np.inf
    q, k, v, g = w.q.copy(), w.k.copy(), w.v.copy(), w.g.copy()
    beta = None if w.beta is None else w.beta.copy()
    state_p = state.copy()
    if kind == "q":
        q[rj, hq, 5] = bad
    elif kind == "k":
        k[rj, hq, 7] = bad
    elif kind == "v":
        v[rj, h, 3] = bad
    elif kind == "g":
        g[rj, h] = bad
    elif kind == "beta":
        beta[rj, h] = bad
    else:
        state_p[1, h, 2, 9] = bad
    wp = dataclasses.replace(w, q=q, k=k, v=v, g=g, beta=beta)
    print(f"non-finite {kind}={bad} case={case} node={j} on_path={on_path}", flush=True)
    out_p, st_p = _run(cfg, wp, state_p)

    heads = group if kind in ("q", "k") else [h]
    T1 = len(parents[1])
    if kind == "q":
        must, may = [j], [j]
    elif kind == "state":
        must, may = list(range(T1)), list(range(T1))
    else:
        must = sub
        spreads = kind == "v" or gdn
        may = list(range(T1)) if spreads else sub
    # other requests and other heads: bit-identical
    rows1 = np.arange(o1, int(w.node_offsets[2]))
    mask = np.ones(out_c.shape, bool)
    for x in heads:
        mask[rows1[may], x, :] = False
    np.testing.assert_array_equal(out_p[mask], out_c[mask])
    for i in must:
        for x in heads:
            assert not np.isfinite(out_p[o1 + i, x]).all(), (kind, i, x)
    # the commit
    smask = np.ones(st_c.shape, bool)
    touched = kind == "state" or (kind != "q" and on_path)
    if touched:
        for x in heads:
            smask[1, x] = False
            assert not np.isfinite(st_p[1, x]).all(), (kind, x)
    np.testing.assert_array_equal(st_p[smask], st_c[smask])
