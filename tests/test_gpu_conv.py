"""GPU parity of the tree-parallel convolution front end (tree_conv_gates) and
the convolution-state commit (tree_conv_state_commit) against the fp64
oracle (oracle/conv_oracle.py), through the C ABI.

Tolerances, from the arithmetic: the kernel computes in fp32 and stores q, k,
v as bf16 with round-to-nearest-even, so an element lies within half a bf16
ulp of the exact value (<= 2^-8 relative) plus the fp32 error of a width-4
dot product, SiLU and a normalisation (~1e-6 of the operands); nearly every
element equals the exact value rounded to bf16 (only values within that fp32
error of a rounding midpoint may go to the other neighbour).  g and beta are
fp32: relative error 1e-5.  The state commit copies bf16 rows: bit-exact."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from synth import workloads as W
from tests import gpu_helpers as H
from paper_2608_01651_amd import treelin as tl

pytestmark = pytest.mark.gpu

CASES = {"tiny": None, "mid": None, "production": [0, 1, 2], "gdn": [0, 1], "large": [0, 1, 2, 3]}


def bf16_cfg(name, **kw):
    cfg = W.CONFIGS[name]
    return dataclasses.replace(cfg, in_dtype="bf16", **kw)


def run_conv(cfg, w, ci, slot=None, num_slots=None, max_nodes=None):
    Hk, Hv, dk, dv = cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v
    prob = H.problem_for(cfg, w.batch, num_slots=num_slots or ci.conv_state.shape[0])
    if max_nodes:
        prob.max_nodes = max_nodes
    N = max(w.N, 1)
    dev = H.dev()
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev).to(torch.bfloat16)
    q = torch.full((N, Hk, dk), float("nan"), device=dev, dtype=torch.bfloat16)
    k = torch.full((N, Hk, dk), float("nan"), device=dev, dtype=torch.bfloat16)
    v = torch.full((N, Hv, dv), float("nan"), device=dev, dtype=torch.bfloat16)
    g = torch.full((N, Hv), float("nan"), device=dev)
    beta = torch.full((N, Hv), float("nan"), device=dev) if cfg.mode == W.GDN else None
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    up_no, up_par = H.t_int(w.node_offsets), H.t_int(w.parent if w.N else np.zeros(1))
    tl.conv_gates(prob, ci.width, up_no, up_par, bf(ci.x if w.N else np.zeros((1, ci.x.shape[1]))),
                  H.t_f32(ci.gate_a if w.N else np.zeros((1, Hv))),
                  None if ci.gate_b is None else H.t_f32(ci.gate_b),
                  H.t_f32(ci.conv_weight), H.t_f32(ci.conv_bias), H.t_f32(ci.A_log),
                  H.t_f32(ci.dt_bias), bf(ci.conv_state), q, k, v, g, beta,
                  slot=None if slot is None else H.t_int(slot), dev_err=err)
    torch.cuda.synchronize()
    out = [t[:w.N].float().cpu().numpy() if t is not None else None for t in (q, k, v, g, beta)]
    return out, int(err.item())


def ref_conv(cfg, w, ci, slot=None):
    return oracle.conv_gates(cfg.mode, cfg.num_qk_heads, cfg.num_v_heads, cfg.d_k, cfg.d_v, ci.width,
                             w.node_offsets, w.parent, ci.x, ci.gate_a, ci.gate_b, ci.conv_weight,
                             ci.conv_bias, ci.A_log, ci.dt_bias, ci.conv_state, slot=slot,
                             max_nodes=cfg.max_nodes)


def check_bf16(got, ref, name, rows=None):
    sel = slice(None) if rows is None else rows
    got, ref = got[sel].astype(np.float64), ref[sel]
    err = np.abs(got - ref)
    bound = 2.0 ** -8 * np.abs(ref) + 1e-5
    assert np.all(err <= bound), f"{name}: worst excess {np.max(err - bound):.3g}"
    rounded = W.round_bf16(ref.astype(np.float32)).astype(np.float64)
    off = np.mean(got != rounded)
    assert off <= 2e-3, f"{name}: {off:.2%} of elements differ from the rounded exact value"


def check_f32(got, ref, name):
    np.testing.assert_allclose(got, ref, rtol=1e-5, atol=1e-6, err_msg=name)


def check_all(out, ref, mode, rows=None):
    for name, a, b in zip(("q", "k", "v"), out[:3], ref[:3]):
        check_bf16(a, b, name, rows)
    sel = slice(None) if rows is None else rows
    check_f32(out[3][sel], ref[3][sel], "g")
    if mode == W.GDN:
        check_f32(out[4][sel], ref[4][sel], "beta")
    else:
        assert out[4] is None


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("width", [4])
def test_conv_gates_parity(name, width):
    cfg = bf16_cfg(name)
    w = W.make(cfg, requests=CASES[name])
    ci = W.make_conv(w, width=width, requests=CASES[name] or range(w.batch))
    out, err = run_conv(cfg, w, ci)
    assert err == 0
    check_all(out, ref_conv(cfg, w, ci), cfg.mode)


@pytest.mark.parametrize("width", [2, 3])
@pytest.mark.parametrize("mode", [W.GLA, W.GDN])
def test_conv_widths_and_modes(width, mode):
    cfg = bf16_cfg("production", mode=mode)
    w = W.make(cfg, requests=[3, 4])
    ci = W.make_conv(w, width=width, requests=[3, 4])
    out, err = run_conv(cfg, w, ci)
    assert err == 0
    check_all(out, ref_conv(cfg, w, ci), mode)


@pytest.mark.parametrize("d, hk, hv", [(16, 2, 4), (32, 3, 3), (64, 1, 4)])
def test_conv_head_dims(d, hk, hv):
    cfg = bf16_cfg("production", d_k=d, d_v=d, num_qk_heads=hk, num_v_heads=hv)
    w = W.make(cfg, requests=[0, 1])
    ci = W.make_conv(w, requests=[0, 1])
    out, err = run_conv(cfg, w, ci)
    assert err == 0
    check_all(out, ref_conv(cfg, w, ci), cfg.mode)


def test_conv_chain_forest_slots_and_empty_requests():
    """A 256-node chain (the window never reaches the state below depth 3), a
    forest with several roots, an empty request, and a slot map."""
    cfg = bf16_cfg("large", num_qk_heads=2, num_v_heads=4)
    rng = np.random.default_rng(7)
    parents = [np.arange(-1, 255, dtype=np.int32), np.array([-1, 0, -1, 2, 1, -1, 5, 6], np.int32),
               np.zeros(0, np.int32)]
    sizes = [len(p) for p in parents]
    base = W.make(cfg, requests=[0, 1, 2])
    w = dataclasses.replace(base, node_offsets=np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32),
                            parent=np.concatenate(parents))
    ci = W.make_conv(w, requests=[0, 1, 2])
    slot = np.array([4, 0, 2], np.int32)
    ci.conv_state = W.round_bf16(rng.standard_normal((5,) + ci.conv_state.shape[1:]).astype(np.float32))
    out, err = run_conv(cfg, w, ci, slot=slot, num_slots=5)
    assert err == 0
    check_all(out, ref_conv(cfg, w, ci, slot=slot), cfg.mode)


def test_conv_device_errors_skip_only_the_bad_request():
    cfg = bf16_cfg("production", num_qk_heads=2, num_v_heads=4)
    w = W.make(cfg, requests=[0, 1, 2])
    ci = W.make_conv(w, requests=[0, 1, 2])
    par = w.parent.copy()
    o1 = int(w.node_offsets[1])
    par[o1 + 5] = 9                                     # a parent after its child
    wb = dataclasses.replace(w, parent=par)
    out, err = run_conv(cfg, wb, ci)
    assert err == tl.TL_EBADTREE
    good = np.r_[0:int(w.node_offsets[1]), int(w.node_offsets[2]):w.N]
    check_all(out, ref_conv(cfg, w, ci), cfg.mode, rows=good)
    o2 = int(w.node_offsets[2])
    assert all(np.isnan(t[o1:o2]).all() for t in out[:4])   # the bad request is not written
    out, err = run_conv(cfg, w, ci, slot=np.array([0, 7, 1], np.int32), num_slots=3)
    assert err == tl.TL_EINVAL


def run_state_commit(cfg, w, ci, terminal, slot=None, num_slots=None):
    prob = H.problem_for(cfg, w.batch, num_slots=num_slots or ci.conv_state.shape[0])
    dev = H.dev()
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev).to(torch.bfloat16)
    cs = bf(ci.conv_state)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    tl.conv_state_commit(prob, ci.width, H.t_int(w.node_offsets), H.t_int(w.parent), H.t_int(terminal),
                         bf(ci.x), cs, slot=None if slot is None else H.t_int(slot), dev_err=err)
    torch.cuda.synchronize()
    return cs.float().cpu().numpy(), int(err.item())


@pytest.mark.parametrize("name", ["production", "gdn", "large"])
@pytest.mark.parametrize("width", [2, 4])
def test_conv_state_commit_bit_exact(name, width):
    cfg = bf16_cfg(name)
    reqs = CASES[name]
    w = W.make(cfg, requests=reqs)
    ci = W.make_conv(w, width=width, requests=reqs)
    term = []
    for b in range(w.batch):                          # the drawn path's terminal; one root; one empty
        p0, p1 = int(w.path_offsets[b]), int(w.path_offsets[b + 1])
        term.append(int(w.path[p1 - 1]) if p1 > p0 else -1)
    term[-1] = -1
    if w.batch > 2:
        term[1] = 0
    term = np.asarray(term, np.int32)
    got, err = run_state_commit(cfg, w, ci, term)
    assert err == 0
    ref = oracle.conv_state_commit(width, w.node_offsets, w.parent, term, ci.x, ci.conv_state,
                                   max_nodes=cfg.max_nodes)
    np.testing.assert_array_equal(got, ref)


def test_conv_state_commit_errors_and_slots():
    cfg = bf16_cfg("production", num_qk_heads=2, num_v_heads=4)
    w = W.make(cfg, requests=[0, 1, 2])
    ci = W.make_conv(w, requests=[0, 1, 2])
    rng = np.random.default_rng(9)
    ci.conv_state = W.round_bf16(rng.standard_normal((4,) + ci.conv_state.shape[1:]).astype(np.float32))
    slot = np.array([3, 1, 0], np.int32)
    term = np.array([5, int(np.diff(w.node_offsets)[1]), 2], np.int32)   # request 1: out of range
    got, err = run_state_commit(cfg, w, ci, term, slot=slot, num_slots=4)
    assert err == tl.TL_EBADPATH
    good = term.copy()
    good[1] = -1
    ref = oracle.conv_state_commit(ci.width, w.node_offsets, w.parent, good, ci.x, ci.conv_state,
                                   slot=slot, max_nodes=cfg.max_nodes)
    np.testing.assert_array_equal(got, ref)
    np.testing.assert_array_equal(got[1], ci.conv_state[1])   # the bad request's slot and slot 2
    np.testing.assert_array_equal(got[2], ci.conv_state[2])
