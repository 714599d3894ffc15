"""GPU tests of the unified cross-layer commit (tree_state_commit_layers) and
the device path export (tree_accepted_path), through the C ABI:

* the exported paths equal the oracle's P(a) = Anc(a) u {a}, bit for bit;
* every layer of one multi-layer launch equals the single-layer commit of
  that layer over the same path, bit for bit, and the fp64 oracle within the
  tolerance;
* device errors skip the bad request in every layer; slot indirection, the
  empty path (terminal -1) and the largest layer count."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from synth import workloads as W
from tests import gpu_helpers as H
from paper_2608_01651_amd import treelin as tl

pytestmark = pytest.mark.gpu

CASES = {"tiny": None, "mid": None, "production": [0, 1, 2, 5], "gdn": [0, 1, 3],
         "large": [0, 1, 2, 3, 4]}


def terminals_of(w):
    """The terminal node of each request's drawn path (-1 when empty)."""
    t = []
    for b in range(w.batch):
        p0, p1 = int(w.path_offsets[b]), int(w.path_offsets[b + 1])
        t.append(int(w.path[p1 - 1]) if p1 > p0 else -1)
    return np.asarray(t, np.int32)


def layer_data(w, n, seed):
    """n layers over w's forest: layer 0 is w itself; the others draw their
    own q/k/v/gates (same distributions, same storage dtype)."""
    cfg = w.cfg
    out = [w]
    for l in range(1, n):
        rng = np.random.default_rng([seed, l, 99])

        def store(x):
            x = np.asarray(x, np.float32)
            return W.round_bf16(x) if cfg.in_dtype == "bf16" else x

        def unit(shape):
            x = rng.standard_normal(shape)
            return store(x / np.linalg.norm(x, axis=-1, keepdims=True))

        N = w.N
        g = (-np.logaddexp(0.0, rng.standard_normal((N, cfg.num_v_heads)) - cfg.gate_shift)).astype(np.float32)
        beta = None
        if cfg.mode == W.GDN:
            beta = (1.0 / (1.0 + np.exp(-rng.standard_normal((N, cfg.num_v_heads))))).astype(np.float32)
        out.append(dataclasses.replace(
            w, q=unit(w.q.shape), k=unit(w.k.shape), v=store(rng.standard_normal(w.v.shape)),
            g=g, beta=beta))
    return out


def rand_state(cfg, slots, seed):
    rng = np.random.default_rng([seed, 555])
    return (0.3 * rng.standard_normal((slots, cfg.num_v_heads, cfg.d_v, cfg.d_k))).astype(np.float32)


def run_layers(cfg, ups, states, terminal, slot=None, num_slots=None):
    prob = H.problem_for(cfg, ups[0].w.batch, num_slots=num_slots or states[0].shape[0])
    err = torch.zeros(1, dtype=torch.int32, device=H.dev())
    tl.commit_layers(prob, [(u.k, u.v, u.g, u.beta, s) for u, s in zip(ups, states)],
                     ups[0].node_offsets, ups[0].parent, H.t_int(terminal), slot=slot, dev_err=err)
    torch.cuda.synchronize()
    return int(err.item())


@pytest.mark.parametrize("name", list(CASES))
def test_accepted_path_bit_exact(name):
    cfg = W.CONFIGS[name]
    w = W.make(name)                                   # full batch
    up = H.Uploaded(w)
    rng = np.random.default_rng(3)
    sizes = np.diff(w.node_offsets)
    term = terminals_of(w)
    for b in range(w.batch):                           # mix in other nodes and empty paths
        if b % 5 == 4:
            term[b] = -1
        elif b % 5 == 3 and sizes[b] > 0:
            term[b] = int(rng.integers(sizes[b]))
    ref_offs, ref_path = oracle.accepted_paths(w.node_offsets, w.parent, term, cfg.max_nodes)
    prob = H.problem_for(cfg, w.batch)
    plen = torch.full((w.batch,), -7, dtype=torch.int32, device=H.dev())
    path = torch.full((max(w.N, 1),), -9, dtype=torch.int32, device=H.dev())
    err = torch.zeros(1, dtype=torch.int32, device=H.dev())
    tl.accepted_path(prob, up.node_offsets, up.parent, H.t_int(term), plen, path, dev_err=err)
    torch.cuda.synchronize()
    assert err.item() == 0
    plen, path = plen.cpu().numpy(), path.cpu().numpy()
    assert plen.tolist() == np.diff(ref_offs).tolist()
    for b in range(w.batch):
        o = int(w.node_offsets[b])
        L = int(plen[b])
        assert path[o:o + L].tolist() == ref_path[ref_offs[b]:ref_offs[b + 1]].tolist()
        assert (path[o + L:int(w.node_offsets[b + 1])] == -9).all()     # the rest is untouched
    # the drawn paths themselves come back for their own terminals
    offs2, path2 = oracle.accepted_paths(w.node_offsets, w.parent, terminals_of(w), cfg.max_nodes)
    assert offs2.tolist() == w.path_offsets.tolist() and path2.tolist() == w.path.tolist()


@pytest.mark.parametrize("name", list(CASES))
def test_commit_layers_parity(name):
    cfg = W.CONFIGS[name]
    w = W.make(name, requests=CASES[name])
    layers = layer_data(w, 3, seed=11)
    ups = [H.Uploaded(x) for x in layers]
    term = terminals_of(w)
    term[-1] = -1 if w.batch > 1 else term[-1]         # one request accepts nothing
    states0 = [rand_state(cfg, w.batch, seed=l) for l in range(3)]
    st_multi = [H.t_f32(s) for s in states0]
    assert run_layers(cfg, ups, st_multi, term) == 0
    # the same layers one launch each, along the exported path
    offs, path = oracle.accepted_paths(w.node_offsets, w.parent, term, cfg.max_nodes)
    prob = H.problem_for(cfg, w.batch)
    for l, (u, s0) in enumerate(zip(ups, states0)):
        single = H.t_f32(s0)
        err = torch.zeros(1, dtype=torch.int32, device=H.dev())
        tl.commit(prob, u.node_offsets, u.parent, H.t_int(offs),
                  H.t_int(path) if path.size else None, u.k, u.v, u.g, u.beta, single, dev_err=err)
        torch.cuda.synchronize()
        assert err.item() == 0
        assert torch.equal(single, st_multi[l]), f"layer {l}: multi-layer launch differs"
    ref = oracle.commit_layers(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, term,
                               [(x.k, x.v, x.g, x.beta, s) for x, s in zip(layers, states0)],
                               max_nodes=cfg.max_nodes)
    for l in range(3):
        got = st_multi[l].cpu().numpy()
        e = H.state_rel_err(got, ref[l])
        assert e < H.TOL, f"layer {l}: max rel err {e:.3g}"
        if w.batch > 1:
            np.testing.assert_array_equal(got[-1], states0[l][-1])    # terminal -1


def test_commit_layers_device_errors_skip_only_the_bad_request():
    cfg = dataclasses.replace(W.CONFIGS["production"], num_qk_heads=2, num_v_heads=4)
    w = W.make(cfg, requests=[0, 1, 2])
    layers = layer_data(w, 2, seed=5)
    ups = [H.Uploaded(x) for x in layers]
    sizes = np.diff(w.node_offsets)
    states0 = [rand_state(cfg, 3, seed=20 + l) for l in range(2)]
    for bad_term, code in ((int(sizes[1]), tl.TL_EBADPATH), (-2, tl.TL_EBADPATH)):
        term = terminals_of(w)
        term[1] = bad_term
        st = [H.t_f32(s) for s in states0]
        assert run_layers(cfg, ups, st, term) == code
        good = term.copy()
        good[1] = -1
        ref = oracle.commit_layers(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, good,
                                   [(x.k, x.v, x.g, x.beta, s) for x, s in zip(layers, states0)],
                                   max_nodes=cfg.max_nodes)
        for l in range(2):
            got = st[l].cpu().numpy()
            np.testing.assert_array_equal(got[1], states0[l][1])
            assert H.state_rel_err(got, ref[l]) < H.TOL
    # a malformed forest: request 2's parent points forward
    par = w.parent.copy()
    o2 = int(w.node_offsets[2])
    par[o2 + 3] = 5
    wb = dataclasses.replace(w, parent=par)
    ub = [H.Uploaded(dataclasses.replace(x, parent=par)) for x in layers]
    st = [H.t_f32(s) for s in states0]
    assert run_layers(cfg, ub, st, terminals_of(wb)) == tl.TL_EBADTREE
    for l in range(2):
        np.testing.assert_array_equal(st[l].cpu().numpy()[2], states0[l][2])
    # and the path export reports the same cases
    prob = H.problem_for(cfg, 3)
    plen = torch.full((3,), -7, dtype=torch.int32, device=H.dev())
    path = torch.full((w.N,), -9, dtype=torch.int32, device=H.dev())
    err = torch.zeros(1, dtype=torch.int32, device=H.dev())
    term = terminals_of(w)
    term[0] = int(sizes[0]) + 3
    tl.accepted_path(prob, ups[0].node_offsets, ups[0].parent, H.t_int(term), plen, path, dev_err=err)
    torch.cuda.synchronize()
    assert err.item() == tl.TL_EBADPATH and plen[0].item() == -7
    assert plen[1:].cpu().tolist() == np.diff(w.path_offsets)[1:].tolist()


def test_commit_layers_slot_indirection():
    cfg = W.CONFIGS["gdn"]
    w = W.make(cfg, requests=[0, 1, 2])
    layers = layer_data(w, 2, seed=8)
    ups = [H.Uploaded(x) for x in layers]
    slot = np.array([4, 0, 2], np.int32)
    states0 = [rand_state(cfg, 5, seed=30 + l) for l in range(2)]
    st = [H.t_f32(s) for s in states0]
    term = terminals_of(w)
    assert run_layers(cfg, ups, st, term, slot=H.t_int(slot), num_slots=5) == 0
    ref = oracle.commit_layers(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, term,
                               [(x.k, x.v, x.g, x.beta, s) for x, s in zip(layers, states0)],
                               slot=slot, max_nodes=cfg.max_nodes)
    for l in range(2):
        got = st[l].cpu().numpy()
        assert H.state_rel_err(got, ref[l]) < H.TOL
        for s in (1, 3):                                   # slots no request names
            np.testing.assert_array_equal(got[s], states0[l][s])


@pytest.mark.parametrize("d", [16, 64])
def test_commit_layers_most_layers(d):
    cfg = dataclasses.replace(W.CONFIGS["mid"], d_k=d, d_v=d, num_qk_heads=1, num_v_heads=2,
                              prefix_len=0)
    w = W.make(cfg, requests=[0])
    n = tl.MAX_COMMIT_LAYERS
    layers = layer_data(w, n, seed=2)
    ups = [H.Uploaded(x) for x in layers]
    states0 = [rand_state(cfg, 1, seed=40 + l) for l in range(n)]
    st = [H.t_f32(s) for s in states0]
    term = terminals_of(w)
    assert run_layers(cfg, ups, st, term) == 0
    ref = oracle.commit_layers(cfg.mode, cfg.num_qk_heads, w.node_offsets, w.parent, term,
                               [(x.k, x.v, x.g, x.beta, s) for x, s in zip(layers, states0)],
                               max_nodes=cfg.max_nodes)
    for l in range(n):
        assert H.state_rel_err(st[l].cpu().numpy(), ref[l]) < H.TOL, f"layer {l}"
